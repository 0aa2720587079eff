// CPU emulation of the HIP runtime and of wave64 SIMT execution (test infrastructure, never
// part of the library), for checking the generated kernels on the host: device memory is host memory placed against
// PROT_NONE guard zones (any access outside a buffer faults at once and is
// reported with the buffer, the offset, the kernel and the thread); every kernel
// thread is a fiber, wave collectives (MFMA, shuffles, ballots, wave barriers)
// and block barriers synchronise the fibers that take part.
#include <dlfcn.h>
#include <execinfo.h>
#include <signal.h>
#include <sys/mman.h>
#include <unistd.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "emu_rt.h"
#include "hip/hip_runtime.h"

// ---------------------------------------------------------------- guarded memory
namespace {
constexpr size_t kPage = 4096;
constexpr size_t kGuard = size_t(1) << 32;   // 4 GiB of PROT_NONE on each side
struct Region { char* base; size_t total; char* start; size_t bytes; std::string tag; int id; bool live; };
std::vector<Region> g_regions;
int g_next_id = 0;
bool start_aligned() { const char* e = getenv("SOBEK_EMU_ALIGN"); return e && e[0] == 's'; }
}  // namespace

extern "C" void* emu_galloc(size_t n, const char* tag) {
  const size_t rn = (n + 15) / 16 * 16 + (n == 0 ? 16 : 0);
  const size_t pages = (rn + kPage - 1) / kPage;
  const size_t total = 2 * kGuard + pages * kPage;
  char* base = (char*)mmap(nullptr, total, PROT_NONE, MAP_PRIVATE | MAP_ANONYMOUS | MAP_NORESERVE, -1, 0);
  if (base == MAP_FAILED) { perror("mmap"); abort(); }
  char* data = base + kGuard;
  if (mprotect(data, pages * kPage, PROT_READ | PROT_WRITE)) { perror("mprotect"); abort(); }
  char* start = start_aligned() ? data : data + pages * kPage - rn;
  memset(data, 0xff, pages * kPage);   // NaN floats, -1 ints: unwritten memory shows
  g_regions.push_back({base, total, start, n, tag ? tag : "?", g_next_id++, true});
  return start;
}

extern "C" void emu_gfree(void* p) {
  for (auto& r : g_regions)
    if (r.live && r.start == p) {
      // keep the range reserved and inaccessible: a later access through a stale pointer faults
      mprotect(r.base, r.total, PROT_NONE);
      r.live = false;
      return;
    }
  if (p) { fprintf(stderr, "emu: free of unknown pointer %p\n", p); abort(); }
}

// ---------------------------------------------------------------- fibers
extern "C" void emu_ctx_switch(void** save_sp, void* to_sp);
extern "C" void emu_fiber_trampoline();
asm(R"(
.text
.globl emu_ctx_switch
.type emu_ctx_switch,@function
emu_ctx_switch:
  pushq %rbp
  pushq %rbx
  pushq %r12
  pushq %r13
  pushq %r14
  pushq %r15
  subq $16, %rsp
  stmxcsr 8(%rsp)
  fnstcw (%rsp)
  movq %rsp, (%rdi)
  movq %rsi, %rsp
  fldcw (%rsp)
  ldmxcsr 8(%rsp)
  addq $16, %rsp
  popq %r15
  popq %r14
  popq %r13
  popq %r12
  popq %rbx
  popq %rbp
  ret
.globl emu_fiber_trampoline
.type emu_fiber_trampoline,@function
emu_fiber_trampoline:
  movq %r12, %rdi
  andq $-16, %rsp
  call emu_fiber_main
  ud2
)");

// AddressSanitizer builds: tell it about the fiber stacks (weak: absent without ASan)
extern "C" {
void __sanitizer_start_switch_fiber(void** fake_stack_save, const void* bottom, size_t size) __attribute__((weak));
void __sanitizer_finish_switch_fiber(void* fake_stack_save, const void** bottom_old, size_t* size_old)
    __attribute__((weak));
void __asan_unpoison_memory_region(void const volatile* addr, size_t size) __attribute__((weak));
}

EmuThread* emu_cur = nullptr;
EmuDim emu_blockIdx, emu_blockDim, emu_gridDim;

namespace {
enum { RUNNABLE, WAIT_WAVE, WAIT_BLOCK, DONE };
struct Fiber {
  void* sp = nullptr;
  void* fake = nullptr;
  char* stack = nullptr;
  EmuThread t{};
  int state = DONE;
  uint64_t wait_gen = 0;
  int site = 0;
};
struct Wave {
  int alive = 0, arrived = 0, site = 0, n = 0;
  uint64_t gen = 0, arr_mask = 0, snap_mask = 0;
  alignas(64) unsigned char dep[64 * 64];
  alignas(64) unsigned char snap[64 * 64];
};
constexpr size_t kStack = 512 * 1024;
std::vector<Fiber> g_fibers;
std::vector<Wave> g_waves;
int g_block_alive = 0, g_block_arrived = 0;
uint64_t g_block_gen = 0;
void* g_sched_sp = nullptr;
void* g_sched_fake = nullptr;
const void* g_sched_bottom = nullptr;
size_t g_sched_size = 0;
Fiber* g_cur = nullptr;
void (*g_entry)(void*) = nullptr;
void* g_ctx = nullptr;
const char* g_kernel = "";
bool g_in_kernel = false;

void complete(Wave& w) {
  memcpy(w.snap, w.dep, sizeof(w.dep));
  w.snap_mask = w.arr_mask;
  w.arr_mask = 0;
  w.arrived = 0;
  w.gen++;
}

void to_scheduler() {
  Fiber* f = g_cur;
  if (__sanitizer_start_switch_fiber) __sanitizer_start_switch_fiber(&f->fake, g_sched_bottom, g_sched_size);
  emu_ctx_switch(&f->sp, g_sched_sp);
  if (__sanitizer_finish_switch_fiber) __sanitizer_finish_switch_fiber(f->fake, &g_sched_bottom, &g_sched_size);
}

void fail_here(const char* what) {
  fprintf(stderr, "emu: %s in kernel %s block (%u,%u,%u) thread %d\n", what, g_kernel, emu_blockIdx.x,
          emu_blockIdx.y, emu_blockIdx.z, emu_cur ? emu_cur->flat : -1);
  fflush(stderr);
  abort();
}
}  // namespace

extern "C" void emu_fiber_main(Fiber* f) {
  if (__sanitizer_finish_switch_fiber) __sanitizer_finish_switch_fiber(nullptr, &g_sched_bottom, &g_sched_size);
  g_entry(g_ctx);
  f->state = DONE;
  Wave& w = g_waves[f->t.wave];
  w.alive--;
  g_block_alive--;
  if (w.arrived > 0 && w.arrived == w.alive) complete(w);
  if (g_block_arrived > 0 && g_block_arrived == g_block_alive) {
    g_block_arrived = 0;
    g_block_gen++;
  }
  if (__sanitizer_start_switch_fiber) __sanitizer_start_switch_fiber(nullptr, g_sched_bottom, g_sched_size);
  emu_ctx_switch(&f->sp, g_sched_sp);
  abort();
}

extern "C" const unsigned char* emu_wave_op(const void* in, int n, int site, uint64_t* mask) {
  Fiber* f = g_cur;
  Wave& w = g_waves[f->t.wave];
  if (w.arrived == 0) {
    w.site = site;
    w.n = n;
  } else if (w.site != site) {
    char b[160];
    snprintf(b, sizeof(b), "divergent wave collective (site %d vs %d, wave %d)", site, w.site, f->t.wave);
    fail_here(b);
  }
  if (n) memcpy(w.dep + 64 * f->t.lane, in, n);
  w.arr_mask |= uint64_t(1) << f->t.lane;
  if (++w.arrived == w.alive) {
    complete(w);
  } else {
    f->state = WAIT_WAVE;
    f->wait_gen = w.gen;
    f->site = site;
    to_scheduler();
  }
  if (mask) *mask = w.snap_mask;
  return w.snap;
}

extern "C" void emu_syncthreads(int site) {
  Fiber* f = g_cur;
  if (++g_block_arrived == g_block_alive) {
    g_block_arrived = 0;
    g_block_gen++;
    return;
  }
  f->state = WAIT_BLOCK;
  f->wait_gen = g_block_gen;
  f->site = site;
  to_scheduler();
}

namespace {
void run_block(int nthreads) {
  if ((int)g_fibers.size() < nthreads) g_fibers.resize(nthreads);
  const int nwaves = (nthreads + 63) / 64;
  if ((int)g_waves.size() < nwaves) g_waves.resize(nwaves);
  for (int wv = 0; wv < nwaves; ++wv) {
    Wave& w = g_waves[wv];
    w.alive = std::min(64, nthreads - 64 * wv);
    w.arrived = 0;
    w.arr_mask = w.snap_mask = 0;
    w.gen = 0;
  }
  g_block_alive = nthreads;
  g_block_arrived = 0;
  g_block_gen = 0;
  for (int i = 0; i < nthreads; ++i) {
    Fiber& f = g_fibers[i];
    if (!f.stack) {
      f.stack = (char*)mmap(nullptr, kStack + kPage, PROT_READ | PROT_WRITE, MAP_PRIVATE | MAP_ANONYMOUS | MAP_NORESERVE,
                            -1, 0);
      if (f.stack == MAP_FAILED) { perror("mmap stack"); abort(); }
      mprotect(f.stack, kPage, PROT_NONE);   // overflow guard
    }
    f.t.flat = i;
    f.t.tid = {(unsigned)(i % emu_blockDim.x), (unsigned)(i / emu_blockDim.x % emu_blockDim.y),
               (unsigned)(i / (emu_blockDim.x * emu_blockDim.y))};
    f.t.lane = i & 63;
    f.t.wave = i >> 6;
    f.state = RUNNABLE;
    if (__asan_unpoison_memory_region) __asan_unpoison_memory_region(f.stack + kPage, kStack);
    uint64_t* top = (uint64_t*)(((uintptr_t)(f.stack + kPage + kStack)) & ~uintptr_t(15));
    uint64_t* sp = top - 10;
    sp[0] = 0x037f;        // x87 control word
    sp[1] = 0x1f80;        // mxcsr
    sp[2] = sp[3] = sp[4] = 0;
    sp[5] = (uint64_t)&f;  // r12: the fiber
    sp[6] = sp[7] = 0;
    sp[8] = (uint64_t)&emu_fiber_trampoline;
    sp[9] = 0;
    f.sp = sp;
  }
  for (;;) {
    bool ran = false, all_done = true;
    for (int i = 0; i < nthreads; ++i) {
      Fiber& f = g_fibers[i];
      if (f.state == DONE) continue;
      all_done = false;
      if (f.state == WAIT_WAVE && g_waves[f.t.wave].gen == f.wait_gen) continue;
      if (f.state == WAIT_BLOCK && g_block_gen == f.wait_gen) continue;
      f.state = RUNNABLE;
      g_cur = &f;
      emu_cur = &f.t;
      if (__sanitizer_start_switch_fiber) __sanitizer_start_switch_fiber(&g_sched_fake, f.stack + kPage, kStack);
      emu_ctx_switch(&g_sched_sp, f.sp);
      if (__sanitizer_finish_switch_fiber) __sanitizer_finish_switch_fiber(g_sched_fake, nullptr, nullptr);
      ran = true;
    }
    if (all_done) break;
    if (!ran) {
      fprintf(stderr, "emu: deadlock in kernel %s block (%u,%u,%u):\n", g_kernel, emu_blockIdx.x, emu_blockIdx.y,
              emu_blockIdx.z);
      for (int i = 0; i < nthreads; ++i)
        if (g_fibers[i].state != DONE)
          fprintf(stderr, "  thread %d state %d site %d\n", i, g_fibers[i].state, g_fibers[i].site);
      abort();
    }
  }
  g_cur = nullptr;
  emu_cur = nullptr;
}

long g_launches = 0;
char* g_lds_b = nullptr;
char* g_lds_e = nullptr;
}  // namespace

extern "C" void emu_set_lds(char* b, char* e) {
  g_lds_b = b;
  g_lds_e = e;
}

extern "C" void emu_run_grid(const char* name, EmuDim grid, EmuDim block, void (*entry)(void*), void* ctx) {
  g_entry = entry;
  g_ctx = ctx;
  g_kernel = name;
  emu_gridDim = grid;
  emu_blockDim = block;
  g_in_kernel = true;
  const int nthreads = (int)(block.x * block.y * block.z);
  if (getenv("SOBEK_EMU_TRACE")) fprintf(stderr, "emu: launch %s grid (%u,%u,%u) block %d\n", name, grid.x, grid.y, grid.z, nthreads);
  // blocks in launch order, or (SOBEK_EMU_ORDER=rev) reversed: results that depend on the order of
  // blocks within one launch show up as differences between the two
  const char* order = getenv("SOBEK_EMU_ORDER");
  const bool rev = order && order[0] == 'r';
  const long nb = (long)grid.x * grid.y * grid.z;
  for (long i = 0; i < nb; ++i) {
    const long b = rev ? nb - 1 - i : i;
    emu_blockIdx = {(unsigned)(b % grid.x), (unsigned)(b / grid.x % grid.y), (unsigned)(b / ((long)grid.x * grid.y))};
    if (g_lds_b && g_lds_e > g_lds_b) memset(g_lds_b, 0xff, g_lds_e - g_lds_b);
    run_block(nthreads);
  }
  g_in_kernel = false;
  g_launches++;
}

extern "C" void emu_note(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vfprintf(stderr, fmt, ap);
  va_end(ap);
}

// ---------------------------------------------------------------- fault reporting
namespace {
void on_segv(int sig, siginfo_t* si, void*) {
  char* a = (char*)si->si_addr;
  fprintf(stderr, "\nemu: %s at address %p", sig == SIGSEGV ? "SIGSEGV" : "SIGBUS", (void*)a);
  if (g_in_kernel)
    fprintf(stderr, " in kernel %s block (%u,%u,%u) thread %d", g_kernel, emu_blockIdx.x, emu_blockIdx.y,
            emu_blockIdx.z, emu_cur ? emu_cur->flat : -1);
  fprintf(stderr, "\n");
  for (auto& r : g_regions)
    if (a >= r.base && a < r.base + r.total) {
      long long off = (long long)(a - r.start);
      fprintf(stderr, "emu:   buffer #%d '%s' (%zu bytes%s): offset %lld (%s)\n", r.id, r.tag.c_str(), r.bytes,
              r.live ? "" : ", freed", off, off < 0 ? "before the start" : "past the end");
    }
  for (auto& f : g_fibers)
    if (f.stack && a >= f.stack && a < f.stack + kPage) fprintf(stderr, "emu:   fiber stack overflow\n");
  void* bt[64];
  int n = backtrace(bt, 64);
  for (int i = 0; i < n; ++i) {
    Dl_info d;
    if (dladdr(bt[i], &d) && d.dli_fname)
      fprintf(stderr, "emu:   #%d %s+0x%lx %s\n", i, d.dli_fname, (long)((char*)bt[i] - (char*)d.dli_fbase),
              d.dli_sname ? d.dli_sname : "");
  }
  fflush(stderr);
  _exit(86);
}
struct SegvInit {
  SegvInit() {
    static char altstack[1 << 16];
    stack_t ss{};
    ss.ss_sp = altstack;
    ss.ss_size = sizeof(altstack);
    sigaltstack(&ss, nullptr);
    struct sigaction sa{};
    sa.sa_sigaction = on_segv;
    sa.sa_flags = SA_SIGINFO | SA_ONSTACK;
    sigaction(SIGSEGV, &sa, nullptr);
    sigaction(SIGBUS, &sa, nullptr);
  }
} g_segv_init;
}  // namespace

// ---------------------------------------------------------------- HIP API
struct EmuModule { void* dl; std::string co; std::map<std::string, std::map<std::string, long>> meta; };
struct EmuFunc {
  std::string name;
  void (*launch)(EmuDim, EmuDim, void**);
  std::map<std::string, long> meta;
};

namespace {
// kernel metadata of the gfx950 code object built from the same source (scratch, VGPRs, LDS)
std::map<std::string, std::map<std::string, long>> read_meta(const std::string& co) {
  std::map<std::string, std::map<std::string, long>> m;
  if (co.empty() || access(co.c_str(), R_OK)) return m;
  std::string cmd = "/opt/rocm/llvm/bin/llvm-readelf --notes '" + co + "' 2>/dev/null";
  FILE* p = popen(cmd.c_str(), "r");
  if (!p) return m;
  char line[512];
  std::vector<std::pair<std::string, long>> pending;
  std::string name;
  auto flush = [&]() {
    if (!name.empty()) for (auto& kv : pending) m[name][kv.first] = kv.second;
    pending.clear();
    name.clear();
  };
  while (fgets(line, sizeof(line), p)) {
    char key[128];
    char val[256];
    if (sscanf(line, " - .args: %127s", key) == 1 || strstr(line, "  - .agpr_count:")) flush();
    if (sscanf(line, " .%127[a-z_]: %255s", key, val) == 2 || sscanf(line, " - .%127[a-z_]: %255s", key, val) == 2) {
      std::string k = key;
      if (k == "name") name = val;
      else if (k == "private_segment_fixed_size" || k == "vgpr_count" || k == "group_segment_fixed_size" ||
               k == "agpr_count" || k == "sgpr_count")
        pending.push_back({k, atol(val)});
    }
  }
  flush();
  pclose(p);
  return m;
}
}  // namespace

extern "C" {
const char* hipGetErrorString(hipError_t e) { return e == hipSuccess ? "no error" : "emulated HIP error"; }
hipError_t hipMalloc(void** p, size_t n) {
  *p = emu_galloc(n, "hipMalloc");
  return hipSuccess;
}
hipError_t hipFree(void* p) {
  emu_gfree(p);
  return hipSuccess;
}
hipError_t hipMemcpy(void* d, const void* s, size_t n, hipMemcpyKind) {
  if (n) memmove(d, s, n);
  return hipSuccess;
}
hipError_t hipMemcpyAsync(void* d, const void* s, size_t n, hipMemcpyKind k, hipStream_t) { return hipMemcpy(d, s, n, k); }
hipError_t hipMemsetAsync(void* d, int v, size_t n, hipStream_t) {
  memset(d, v, n);
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
// Launches run to completion in call order, so every stream is one stream and events order nothing
// further; a created stream is a distinct non-null handle.
hipError_t hipStreamCreateWithFlags(hipStream_t* s, unsigned) {
  static int side;
  *s = &side;
  return hipSuccess;
}
hipError_t hipStreamDestroy(hipStream_t) { return hipSuccess; }
hipError_t hipStreamWaitEvent(hipStream_t, hipEvent_t, unsigned) { return hipSuccess; }
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned) { return hipEventCreate(e); }
hipError_t hipEventCreate(hipEvent_t* e) {
  static int dummy;
  *e = &dummy;
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }
hipError_t hipEventSynchronize(hipEvent_t) { return hipSuccess; }
hipError_t hipEventElapsedTime(float* ms, hipEvent_t, hipEvent_t) {
  *ms = 0.f;
  return hipSuccess;
}
hipError_t hipEventDestroy(hipEvent_t) { return hipSuccess; }
// image: "<cpu shared object>\n<gfx950 code object or empty>\0"
hipError_t hipModuleLoadData(hipModule_t* m, const void* image) {
  std::string s((const char*)image);
  auto nl = s.find('\n');
  std::string so = s.substr(0, nl), co = nl == std::string::npos ? "" : s.substr(nl + 1);
  void* dl = dlopen(so.c_str(), RTLD_NOW | RTLD_LOCAL);
  if (!dl) {
    fprintf(stderr, "emu: dlopen %s: %s\n", so.c_str(), dlerror());
    return hipErrorInvalidValue;
  }
  *m = new EmuModule{dl, co, read_meta(co)};
  return hipSuccess;
}
hipError_t hipModuleUnload(hipModule_t) { return hipSuccess; }
hipError_t hipModuleGetFunction(hipFunction_t* f, hipModule_t m, const char* name) {
  std::string sym = std::string(name) + "__cpu";
  void* p = dlsym(m->dl, sym.c_str());
  if (!p) {
    fprintf(stderr, "emu: no kernel %s\n", name);
    return hipErrorNotFound;
  }
  auto it = m->meta.find(name);
  *f = new EmuFunc{name, (void (*)(EmuDim, EmuDim, void**))p, it == m->meta.end() ? std::map<std::string, long>{} : it->second};
  return hipSuccess;
}
hipError_t hipModuleLaunchKernel(hipFunction_t f, unsigned gx, unsigned gy, unsigned gz, unsigned bx, unsigned by,
                                 unsigned bz, unsigned shmem, hipStream_t, void** params, void**) {
  const long lds = f->meta.count("group_segment_fixed_size") ? f->meta["group_segment_fixed_size"] : -1;
  if (lds + (long)shmem > 160 * 1024) {
    fprintf(stderr, "emu: kernel %s needs %ld bytes of LDS\n", f->name.c_str(), lds + shmem);
    return hipErrorLaunchFailure;
  }
  if (bx * by * bz > 1024 || bx * by * bz == 0) {
    fprintf(stderr, "emu: kernel %s block of %u threads\n", f->name.c_str(), bx * by * bz);
    return hipErrorLaunchFailure;
  }
  if (gy > 65535 || gz > 65535) {
    fprintf(stderr, "emu: kernel %s grid (%u,%u,%u)\n", f->name.c_str(), gx, gy, gz);
    return hipErrorLaunchFailure;
  }
  f->launch(EmuDim{gx, gy, gz}, EmuDim{bx, by, bz}, params);
  return hipSuccess;
}
hipError_t hipFuncGetAttribute(int* v, hipFunction_attribute a, hipFunction_t f) {
  auto get = [&](const char* k, long d) { return f->meta.count(k) ? f->meta[k] : d; };
  switch (a) {
    case HIP_FUNC_ATTRIBUTE_LOCAL_SIZE_BYTES: *v = (int)get("private_segment_fixed_size", 0); break;
    case HIP_FUNC_ATTRIBUTE_NUM_REGS: *v = (int)get("vgpr_count", 64); break;
    case HIP_FUNC_ATTRIBUTE_SHARED_SIZE_BYTES: *v = (int)get("group_segment_fixed_size", 0); break;
    default: *v = 0;
  }
  if (getenv("SOBEK_EMU_TRACE")) fprintf(stderr, "emu: attribute %d of %s = %d\n", (int)a, f->name.c_str(), *v);
  return hipSuccess;
}
hipError_t hipGetDevice(int* d) {
  *d = 0;
  return hipSuccess;
}
hipError_t hipGetSymbolAddress(void** p, const EmuSymbol* sym) {
  static std::map<const EmuSymbol*, void*> m;
  if (!m.count(sym)) m[sym] = emu_galloc(sym->bytes, "static scratch");
  *p = m[sym];
  return hipSuccess;
}
long emu_launch_count() { return g_launches; }
}
