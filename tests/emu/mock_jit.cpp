// Plan compiler of the CPU emulation build (test infrastructure, never part of the library):
// the generated source (prelude + plan) is compiled for the host against emu_device.h into a
// shared object, cached by content hash; the module image handed to hipModuleLoadData names
// that object and the gfx950 code object the real library loads for the same source, whose
// metadata (LDS, scratch and register use) the emulated runtime reports and checks.
#include <fcntl.h>
#include <sys/file.h>
#include <sys/stat.h>
#include <unistd.h>

#include <dlfcn.h>

#include <cstdio>
#include <cstdlib>
#include <fstream>
#include <regex>
#include <set>
#include <sstream>
#include <stdexcept>
#include <string>
#include <vector>

#include "../../paper_2607_18074_amd/csrc/jit.h"

namespace sobek {
namespace {
const char* kPrelude =
#include "../../paper_2607_18074_amd/csrc/prelude_embed.inc"
    ;
const std::vector<std::string>& options() {
  static const std::vector<std::string> o = {"--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang",
                                             "-target-feature", "-Xclang", "-packed-fp32-ops"};
  return o;
}
uint64_t fnv1a(const std::string& s, uint64_t h = 1469598103934665603ull) {
  for (unsigned char c : s) {
    h ^= c;
    h *= 1099511628211ull;
  }
  return h;
}
std::string env_or(const char* k, const std::string& d) {
  const char* e = getenv(k);
  return e && *e ? e : d;
}
// directory of the emulation library (the build directory)
std::string lib_dir() {
  Dl_info info;
  if (dladdr((void*)&fnv1a, &info) && info.dli_fname) {
    std::string p = info.dli_fname;
    auto pos = p.find_last_of('/');
    if (pos != std::string::npos) return p.substr(0, pos);
  }
  return ".";
}
}  // namespace

std::string full_source(const std::string& plan_source) { return std::string(kPrelude) + plan_source; }

std::string jit_key(const std::string& plan_source) {
  uint64_t h = fnv1a(full_source(plan_source));
  for (auto& o : options()) h = fnv1a(o, h);
  char b[32];
  snprintf(b, sizeof(b), "%016llx", (unsigned long long)h);
  return b;
}

std::vector<char> jit_compile(const std::string& plan_source, std::string* log) {
  // build directory (library, kernel cache), emulator sources (headers), real code-object cache
  const std::string lib = env_or("SOBEK_EMU_LIBDIR", lib_dir());
  const std::string emu = env_or("SOBEK_EMU_SRC", lib + "/..");
  const std::string gpu_cache = env_or("SOBEK_EMU_GPU_CACHE", emu + "/../../paper_2607_18074_amd/_jitcache");
  const std::string key = jit_key(plan_source);
  const std::string co = gpu_cache + "/sobek_" + key + ".co";
  std::string src = full_source(plan_source);
  // big plans compile for minutes at -O1: those at -O0
  const bool asan = getenv("SOBEK_EMU_ASAN") && getenv("SOBEK_EMU_ASAN")[0] == '1';
  const std::string opt = env_or("SOBEK_EMU_OPT", src.size() > 1500000 ? "-O0" : "-O1") +
                          (asan ? " -fsanitize=address -fno-omit-frame-pointer" : "");
  const std::string libdir = lib;
  // host build key: the source and the emulator header
  std::ifstream hf(emu + "/emu_device.h");
  std::stringstream hs;
  hs << hf.rdbuf();
  char hk[32];
  snprintf(hk, sizeof(hk), "%016llx", (unsigned long long)fnv1a(src, fnv1a(hs.str() + opt + "patches v3")));
  const std::string dir = lib + (asan ? "/cache_asan" : "/cache");
  mkdir(dir.c_str(), 0755);
  const std::string so = dir + "/k_" + hk + ".so";
  // one compile per plan across processes: the others wait on the lock, then load its result
  const int lockfd = open((so + ".lock").c_str(), O_CREAT | O_RDWR, 0644);
  if (lockfd >= 0) flock(lockfd, LOCK_EX);
  struct Unlock {
    int fd;
    ~Unlock() {
      if (fd >= 0) { flock(fd, LOCK_UN); close(fd); }
    }
  } unlock{lockfd};
  if (access(so.c_str(), R_OK)) {
    // amdgpu-only kernel attributes
    const std::string attr = "__attribute__((amdgpu_waves_per_eu(";
    for (size_t at = src.find(attr); at != std::string::npos; at = src.find(attr, at)) {
      size_t e = src.find(")))", at);
      src.erase(at, e + 3 - at);
    }
    // wave-lockstep points the hardware gives implicitly: after the per-wave sender-id staging and
    // before a forward unit rewrites its coupling table (the emulated lanes run one after another
    // between wave collectives)
    {
      std::istringstream in(src);
      std::ostringstream out;
      std::string line;
      while (std::getline(in, line)) {
        if (line.find("const float rinv = __builtin_amdgcn_rsqf(evx * evx") != std::string::npos)
          out << "emu_wave_sync(__LINE__);\n";
        out << line << "\n";
        if (line.find("ids[64 * i + lane] = sender[") != std::string::npos) out << "emu_wave_sync(__LINE__);\n";
      }
      src = out.str();
    }
    const std::string base = dir + "/k_" + hk;
    std::ofstream(base + ".cpp") << "#include \"emu_device.h\"\n" << src << "\n";
    // kernel names after macro expansion (token-pasted names included)
    std::string pp = "/opt/rocm/llvm/bin/clang++ -std=c++17 -E -DEMU_SCAN -I" + emu + " " + base + ".cpp -o " + base +
                     ".ii 2> " + base + ".log";
    if (system(pp.c_str()) != 0) throw std::runtime_error("host preprocessing of the plan failed");
    std::ifstream pf(base + ".ii");
    std::stringstream ps;
    ps << pf.rdbuf();
    const std::string ii = ps.str();
    std::set<std::string> names;
    const std::string mark = "EMU_GLOBAL_MARK";
    for (size_t at = ii.find(mark); at != std::string::npos; at = ii.find(mark, at + 1)) {
      size_t v = ii.find("void ", at);
      size_t b = v + 5, e = ii.find('(', b);
      std::string n = ii.substr(b, e - b);
      while (!n.empty() && n.back() == ' ') n.pop_back();
      if (n.find(' ') == std::string::npos && !n.empty()) names.insert(n);
    }
    std::ostringstream o;
    o << "#include \"emu_device.h\"\n" << src << "\n";
    for (auto& n : names)
      o << "extern \"C\" void " << n << "__cpu(EmuDim g, EmuDim b, void** p) { emu_launch(\"" << n << "\", " << n
        << ", g, b, p); }\n";
    const std::string cpp = base + ".cpp";
    std::ofstream(cpp) << o.str();
    const std::string tmp = so + ".tmp" + std::to_string(getpid());
    std::string cmd = "/opt/rocm/llvm/bin/clang++ -std=c++17 " + opt +
                      " -g -fPIC -shared -w -I" + emu + " -o " + tmp + " " + cpp + " -L" + libdir +
                      " -lsobek_emu -Wl,-rpath," + libdir + " 2> " + dir + "/k_" + hk + ".log";
    fprintf(stderr, "emu: compiling %zu kernels for the host (%s)\n", names.size(), hk);
    if (system(cmd.c_str()) != 0) {
      std::ifstream lf(dir + "/k_" + hk + ".log");
      std::stringstream ls;
      ls << lf.rdbuf();
      if (log) *log = ls.str();
      throw std::runtime_error("host compile of the plan failed: " + ls.str().substr(0, 3000));
    }
    rename(tmp.c_str(), so.c_str());
  }
  std::string img = so + "\n" + (access(co.c_str(), R_OK) ? std::string() : co);
  if (img.find('\n') == img.size() - 1 && getenv("SOBEK_EMU_TRACE"))
    fprintf(stderr, "emu: no gfx950 code object %s\n", co.c_str());
  return std::vector<char>(img.begin(), img.end() + 1);
}

}  // namespace sobek
