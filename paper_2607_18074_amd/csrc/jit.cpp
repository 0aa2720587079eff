// hipRTC compilation of generated plans for gfx950, with a content-addressed
// code-object cache on disk (SOBEK_JIT_CACHE, default: _jitcache/ next to the
// library).  The cache key covers the full source and the compile options.
#include <dlfcn.h>
#include <hip/hiprtc.h>
#include <sys/stat.h>
#include <unistd.h>
#include <utime.h>

#include <cstdio>
#include <cstdlib>
#include <fstream>
#include <mutex>
#include <sstream>
#include <stdexcept>
#include <string>
#include <vector>

#include "jit.h"

namespace sobek {

namespace {
const char* kPrelude =
#include "prelude_embed.inc"
    ;

const std::vector<std::string>& options() {
  static const std::vector<std::string> o = {
      "--offload-arch=gfx950", "-O3", "-std=c++17",
      // packed FP32 instructions are not used (plain fp32 VALU and MFMA only)
      "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"};
  return o;
}

uint64_t fnv1a(const std::string& s, uint64_t h = 1469598103934665603ull) {
  for (unsigned char c : s) {
    h ^= c;
    h *= 1099511628211ull;
  }
  return h;
}

std::string lib_dir() {
  Dl_info info;
  if (dladdr((void*)&fnv1a, &info) && info.dli_fname) {
    std::string p = info.dli_fname;
    auto pos = p.find_last_of('/');
    if (pos != std::string::npos) return p.substr(0, pos);
  }
  return ".";
}

std::string cache_dir() {
  const char* env = std::getenv("SOBEK_JIT_CACHE");
  std::string d = env && *env ? env : lib_dir() + "/_jitcache";
  mkdir(d.c_str(), 0755);
  return d;
}

bool read_file(const std::string& path, std::vector<char>& out) {
  std::ifstream f(path, std::ios::binary);
  if (!f) return false;
  out.assign(std::istreambuf_iterator<char>(f), std::istreambuf_iterator<char>());
  return !out.empty();
}

std::mutex g_jit_mu;
}  // namespace

std::string full_source(const std::string& plan_source) { return std::string(kPrelude) + plan_source; }

std::string jit_key(const std::string& plan_source) {
  std::string all = full_source(plan_source);
  uint64_t h = fnv1a(all);
  for (auto& o : options()) h = fnv1a(o, h);
  char b[32];
  std::snprintf(b, sizeof(b), "%016llx", (unsigned long long)h);
  return b;
}

std::vector<char> jit_compile(const std::string& plan_source, std::string* log_out) {
  std::lock_guard<std::mutex> lk(g_jit_mu);
  const std::string key = jit_key(plan_source);
  const std::string path = cache_dir() + "/sobek_" + key + ".co";
  std::vector<char> code;
  if (read_file(path, code)) {
    utime(path.c_str(), nullptr);  // a hit marks the entry as in use (build steps prune untouched ones)
    return code;
  }

  std::string src = full_source(plan_source);
  hiprtcProgram prog;
  if (hiprtcCreateProgram(&prog, src.c_str(), "sobek_plan.hip", 0, nullptr, nullptr) != HIPRTC_SUCCESS)
    throw std::runtime_error("hiprtcCreateProgram failed");
  std::vector<const char*> opts;
  for (auto& o : options()) opts.push_back(o.c_str());
  hiprtcResult r = hiprtcCompileProgram(prog, (int)opts.size(), opts.data());
  size_t ls = 0;
  hiprtcGetProgramLogSize(prog, &ls);
  std::string log(ls, '\0');
  if (ls) hiprtcGetProgramLog(prog, &log[0]);
  if (log_out) *log_out = log;
  if (r != HIPRTC_SUCCESS) {
    hiprtcDestroyProgram(&prog);
    if (std::getenv("SOBEK_JIT_DUMP")) {
      std::ofstream(cache_dir() + "/failed_" + key + ".hip") << src;
    }
    throw std::runtime_error("hipRTC compilation failed: " + log.substr(0, 4000));
  }
  size_t cs = 0;
  hiprtcGetCodeSize(prog, &cs);
  code.resize(cs);
  hiprtcGetCode(prog, code.data());
  hiprtcDestroyProgram(&prog);
  // atomic publish: write to a unique temporary, then rename
  std::string tmp = path + ".tmp" + std::to_string(getpid());
  {
    std::ofstream f(tmp, std::ios::binary);
    f.write(code.data(), (std::streamsize)code.size());
  }
  std::rename(tmp.c_str(), path.c_str());
  if (std::getenv("SOBEK_JIT_DUMP")) std::ofstream(cache_dir() + "/sobek_" + key + ".hip") << src;
  return code;
}

}  // namespace sobek
