// C ABI of libsobek_hip and the host runtime that sequences the generated
// kernels over bounded receiver chunks (Section 4, Appendix B.2).
//
// Receiver-factorised program per chunk of receivers [r0, r0 + n):
//   forward  (Section 4.2):  S = sum_e phi_e (x) C(x_j, Y_e)   [sobek_fwd_S]
//                            m_g = S_g A_g                      [sobek_gemm_sa, per output group]
//   backward (Section 4.3):  Sbar_g = mbar_g A_g^T              [sobek_gemm_sbar]
//                            A_bar_g += S_g^T mbar_g            [sobek_gemm_ga + sobek_ga_reduce]
//                            phi_bar, evec_bar, per-edge x contributions   [sobek_bwd_E]
//                            x_bar via the sender-sorted view   [sobek_sender_reduce]
//   double backward (Section 4.4, eq. receiver_double_adjoint with d mbar = 0):
//                            dS (directional state)             [sobek_fwd_dS]
//                            m_dot = dS A + S dA                [sobek_gemm_sa x2]
//                            Sbar = mbar A^T, Sbar' = mbar dA^T [sobek_gemm_sbar x2]
//                            g_A = dS^T mbar                    [sobek_gemm_ga]
//                            edge-local second adjoints         [sobek_dbwd_E]
//                            g_x via the sender-sorted view     [sobek_sender_reduce]
// Every reduction has a fixed order (CSR order, split order, chunk order), so
// results are bitwise reproducible for a given workspace size.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <stdexcept>
#include <string>
#include <vector>

#include "../../include/sobek.h"
#include "jit.h"
#include "plan.h"
#include "tables.h"

using sobek::Plan;

struct sobek_plan_s {
  Plan p;
  // A second stream for channel GEMMs that overlap the edge stage of the same call, forked from and
  // joined back into the caller's stream with events (created on first use, default priority).
  std::mutex side_mu;
  hipStream_t side = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};

struct sobek_graph_s {
  int64_t N = 0, E = 0;
  const int32_t* rowptr = nullptr;
  const int32_t* sender = nullptr;
  int32_t* send_rowptr = nullptr;
  int32_t* send_perm = nullptr;
  std::vector<int32_t> h_rowptr;
  int64_t max_deg = 0;
};

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[2048];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIPCHK(call)                                                                          \
  do {                                                                                        \
    hipError_t e_ = (call);                                                                   \
    if (e_ != hipSuccess) return fail(SOBEK_E_HIP, "%s: %s", #call, hipGetErrorString(e_));  \
  } while (0)

// Optional instrumentation: when enabled, every launch is bracketed by two
// hipEvents recorded on the launch stream; durations are resolved on query.
struct ProfRec {
  std::string name;
  hipEvent_t a, b;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::map<hipFunction_t, std::string> g_names;
std::vector<ProfRec> g_prof;
std::vector<hipEvent_t> g_event_pool;

hipEvent_t pool_event() {
  if (!g_event_pool.empty()) {
    hipEvent_t e = g_event_pool.back();
    g_event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  (void)hipEventCreate(&e);
  return e;
}

template <typename... Args>
hipError_t launch_n(hipFunction_t f, unsigned nthreads, unsigned gx, unsigned gy, unsigned gz, hipStream_t s,
                    Args... args) {
  if (gx == 0 || gy == 0 || gz == 0) return hipSuccess;
  void* ptrs[] = {(void*)&args...};
  if (!g_prof_on) return hipModuleLaunchKernel(f, gx, gy, gz, nthreads, 1, 1, 0, s, ptrs, nullptr);
  std::lock_guard<std::mutex> lk(g_prof_mu);
  ProfRec r;
  auto it = g_names.find(f);
  r.name = it == g_names.end() ? std::string("?") : it->second;
  r.a = pool_event();
  r.b = pool_event();
  (void)hipEventRecord(r.a, s);
  hipError_t e = hipModuleLaunchKernel(f, gx, gy, gz, nthreads, 1, 1, 0, s, ptrs, nullptr);
  (void)hipEventRecord(r.b, s);
  g_prof.push_back(r);
  return e;
}

template <typename... Args>
hipError_t launch(hipFunction_t f, unsigned gx, unsigned gy, unsigned gz, hipStream_t s, Args... args) {
  return launch_n(f, 256, gx, gy, gz, s, args...);
}

#define LAUNCH(...) HIPCHK(launch(__VA_ARGS__))
#define LAUNCH_N(...) HIPCHK(launch_n(__VA_ARGS__))

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
unsigned cdiv(int64_t a, int64_t b) { return (unsigned)((a + b - 1) / b); }

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

int validate_irreps(const sobek_irrep* v, int n, std::vector<sobek::Irrep>& out, const char* what) {
  if (n <= 0 || !v) return fail(SOBEK_E_INVALID, "%s irreps: empty or NULL", what);
  for (int i = 0; i < n; ++i) {
    if (v[i].mul < 1) return fail(SOBEK_E_INVALID, "%s irrep %d: multiplicity %d < 1", what, i, v[i].mul);
    if (v[i].l < 0) return fail(SOBEK_E_INVALID, "%s irrep %d: negative order", what, i);
    if (v[i].l > 3) return fail(SOBEK_E_UNSUPPORTED, "%s irrep %d: order %d > 3 not supported", what, i, v[i].l);
    if (v[i].parity != 1 && v[i].parity != -1)
      return fail(SOBEK_E_INVALID, "%s irrep %d: parity must be +1 or -1", what, i);
    out.push_back({v[i].mul, v[i].l, v[i].parity, 0});
  }
  return SOBEK_OK;
}

int build_signature(const sobek_irrep* in, int n_in, int lmax, const sobek_irrep* out, int n_out, int K, int mode,
                    int layout, int dtype, int norm, Plan& p) {
  int rc;
  if ((rc = validate_irreps(in, n_in, p.in, "input")) != SOBEK_OK) return rc;
  if ((rc = validate_irreps(out, n_out, p.out, "output")) != SOBEK_OK) return rc;
  if (lmax < 0) return fail(SOBEK_E_INVALID, "lmax < 0");
  if (lmax > 3) return fail(SOBEK_E_UNSUPPORTED, "lmax %d > 3 not supported", lmax);
  if (K < 1 || K > 64) return fail(SOBEK_E_INVALID, "K = %d outside [1, 64]", K);
  if (layout != SOBEK_LAYOUT_IR_MUL && layout != SOBEK_LAYOUT_MUL_IR) return fail(SOBEK_E_INVALID, "bad layout");
  if (dtype != SOBEK_DTYPE_F32 && dtype != SOBEK_DTYPE_BF16_GEMM) return fail(SOBEK_E_INVALID, "bad dtype");
  if (dtype == SOBEK_DTYPE_BF16_GEMM && mode != SOBEK_MODE_UVW)
    return fail(SOBEK_E_UNSUPPORTED, "SOBEK_DTYPE_BF16_GEMM is implemented for uvw plans only");
  if (norm != SOBEK_NORM_NONE && norm != SOBEK_NORM_FAN_IN) return fail(SOBEK_E_INVALID, "bad path normalisation");
  if (mode != SOBEK_MODE_UVW && mode != SOBEK_MODE_UVU) return fail(SOBEK_E_INVALID, "bad mode");
  p.lmax = lmax; p.K = K; p.layout = layout; p.dtype = dtype; p.norm = norm; p.mode = mode;
  try {
    sobek::build_plan(p);
  } catch (const std::invalid_argument& ex) {
    return fail(SOBEK_E_INVALID, "plan: %s", ex.what());
  } catch (const std::exception& ex) {
    return fail(SOBEK_E_UNSUPPORTED, "plan: %s", ex.what());
  }
  if (p.paths.empty()) return fail(SOBEK_E_INVALID, "no path satisfies the selection rules");
  if (dtype == SOBEK_DTYPE_BF16_GEMM && !p.vec4)
    return fail(SOBEK_E_UNSUPPORTED, "SOBEK_DTYPE_BF16_GEMM needs every multiplicity a multiple of 4");
  // SOBEK_UVU_ROUTE=receiver keeps channelwise plans on the receiver-state route (testing and
  // comparison); the state-free kernels are then not generated
  if (const char* r = std::getenv("SOBEK_UVU_ROUTE"))
    if (std::strcmp(r, "receiver") == 0) { p.uvu_C = 0; p.uvu_NB = 0; }
  int64_t maxD = 0;
  for (auto& g : p.groups) maxD = std::max(maxD, g.D);
  if (p.n_w * (int64_t)K >= (1ll << 31) || maxD >= (1ll << 31))
    return fail(SOBEK_E_UNSUPPORTED, "weight tensor too large for 32-bit indexing");
  p.source = sobek::generate_source(p);
  if (p.mode == SOBEK_MODE_UVU && p.uvu_C > 0) p.source_u = sobek::generate_source(p, false);
  return SOBEK_OK;
}

// ----------------------------------------------------------------------------
// workspace planning
// ----------------------------------------------------------------------------
struct Chunk {
  int r0, n;
  int64_t e0, e1;
};

struct WsPlan {
  // byte offsets
  size_t off_x = 0, off_gout = 0, off_tgx = 0, off_out = 0, off_gx = 0, off_cursor = 0, off_P = 0, off_state = 0,
         off_contrib = 0, off_K = 0;
  size_t kfloats = 0;  // split-K partials of the state GEMM (forward and double backward)
  size_t fixed = 0;
  int nstate = 0;
  int64_t ncap = 0, ecap = 0;
  size_t total = 0;
  std::vector<Chunk> chunks;
};

int gemm_bn(int C) { return C <= 16 ? 16 : (C <= 32 ? 32 : 64); }
int bn_index(int bn) { return bn == 16 ? 0 : (bn == 32 ? 1 : 2); }

// Column-tile width of the state GEMM m = S A for a group: bf16-GEMM plans take 128-wide tiles for
// groups wider than 64 channels, so that each block reads its rows of S once instead of once per 64
// columns (Wide forward: 16.7 -> 15.9 ms).  The weight-gradient GEMM keeps 64-wide tiles: with 128
// its split count doubles to keep the GPU busy and the larger partials cost more than the saved reads.
int state_gemm_bn(const Plan& p, const sobek::Group& g) {
  return p.dtype == SOBEK_DTYPE_BF16_GEMM && p.vec4 && g.C > 64 ? 128 : gemm_bn(g.C);
}

int nsplit_for(const Plan& p, const sobek::Group& g, int64_t nrows) {
  const bool vec4 = p.vec4;
  int bn = gemm_bn(g.C);
  int64_t tiles = (int64_t)cdiv(g.D, vec4 ? 128 : 64) * cdiv(g.C, bn);
  int64_t ns = (512 + tiles - 1) / tiles;
  ns = std::max<int64_t>(1, std::min<int64_t>(ns, 64));
  ns = std::min<int64_t>(ns, std::max<int64_t>(1, nrows / 64));
  return (int)ns;
}

// split partials of the weight-gradient GEMMs: one region per output group,
// accumulated over the receiver chunks of a pass and reduced once at its end
size_t partial_floats(const Plan& p, int64_t ncap, int pass = SOBEK_PASS_BWD, int nstate = -1) {
  // the state-free channelwise weight gradient: one partial row of K * N_w floats per wave
  // (the backward, and a double backward planned without receiver state, take that route)
  const bool free = p.mode == SOBEK_MODE_UVU && p.uvu_bwd_direct && p.uvu_wgrad_direct;
  if ((pass == SOBEK_PASS_BWD || (pass == SOBEK_PASS_DBWD && nstate == 0)) && free)
    return (size_t)sobek::uvu_wgrad_waves(p.K, p.n_w) * p.K * p.n_w;
  size_t m = 0;
  for (auto& g : p.groups) m += (size_t)nsplit_for(p, g, ncap * g.d) * g.D * g.C;
  return m;
}

// Split-K of the state GEMM m_g = S_g A_g: a chunk of few receivers gives few row
// tiles against a long reduction (K times the summed input multiplicities), so the
// reduction is split until about kSaTarget blocks run; partial tiles are summed in
// split order by sobek_sa_reduce.  The partials of one group at a time live in a
// region of at most kSaSplitCap floats.
constexpr int kSaTarget = 512, kSaMaxSplit = 16;
constexpr size_t kSaSplitCap = (size_t)4 << 20;

size_t sa_split_floats(const Plan& p, int pass, int64_t ncap) {
  if (pass == SOBEK_PASS_BWD || !p.vec4 || p.mode == SOBEK_MODE_UVU) return 0;
  size_t m = 0;
  for (auto& g : p.groups) m = std::max(m, (size_t)g.d * g.C);
  return std::min(kSaSplitCap, (size_t)kSaMaxSplit * (size_t)std::max<int64_t>(1, ncap) * m);
}

// splits of one state-GEMM launch over nrows rows (1 = no split); kper = reduction per split
int sa_nsplit(const Plan& p, const sobek::Group& g, int64_t nrows, size_t kfloats, int& kper) {
  const int bn = state_gemm_bn(p, g);
  const int64_t blocks = (int64_t)cdiv(nrows, 128) * cdiv(g.C, bn);
  kper = (int)g.D;
  if (blocks * 2 > kSaTarget || nrows <= 0) return 1;
  int64_t ns = std::min<int64_t>({(kSaTarget + blocks - 1) / blocks, (int64_t)kSaMaxSplit,
                                  (int64_t)(kfloats / ((size_t)nrows * g.C)), (int64_t)g.D / (4 * 32)});
  if (ns < 2) return 1;
  kper = (int)(cdiv(cdiv(g.D, ns), 32) * 32);
  return (int)cdiv(g.D, kper);
}

// floats per edge of the state-free channelwise backward's per-block partial sums
// (phi_bar and Y_bar of every 64-channel block), kept after the window's contributions
int64_t uvu_edge_partials(const Plan& p, int pass) {
  const int64_t npart = (int64_t)p.uvu_NB * (p.uvu_sliced ? p.uvu_NA : 1);
  return (pass != SOBEK_PASS_FWD && p.mode == SOBEK_MODE_UVU && p.uvu_bwd_direct && npart > 1)
             ? npart * (p.K + p.nsh)
             : 0;
}

// fixed part + per-receiver + per-edge bytes of a pass
void pass_costs(const Plan& p, const sobek_graph_s& G, int pass, int nstate, WsPlan& w, size_t& per_recv,
                size_t& per_edge) {
  const bool mulir = p.layout == SOBEK_LAYOUT_MUL_IR;
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t at = o; o = align_up(o + bytes); return at; };
  const size_t nx = (size_t)G.N * p.dim_in * 4, no = (size_t)G.N * p.dim_out * 4;
  if (mulir) {
    w.off_x = take(nx);
    w.off_out = take(no);
    if (pass >= SOBEK_PASS_BWD) { w.off_gout = take(no); w.off_gx = take(nx); }
    if (pass == SOBEK_PASS_DBWD) w.off_tgx = take(nx);
  }
  if (pass != SOBEK_PASS_FWD) w.off_cursor = take((size_t)(G.N + 1) * 4);  // per-sender chunk cursors
  w.off_P = o;  // partials, sized once the chunk capacity is known
  w.fixed = o;
  // receiver-state slots: one, reused phase by phase (S, then Sbar); the double
  // backward needs a second one for Sbar' when dA is active
  w.nstate = nstate >= 0 ? nstate : (pass == SOBEK_PASS_DBWD ? 2 : 1);
  // the state-free channelwise forward keeps no receiver state (a kept one is the caller's)
  if (pass == SOBEK_PASS_FWD && p.mode == SOBEK_MODE_UVU && p.uvu_C > 0) w.nstate = 0;
  per_recv = (size_t)w.nstate * p.srow * 4;
  per_edge = pass == SOBEK_PASS_FWD ? 0 : (size_t)(p.dim_in + uvu_edge_partials(p, pass)) * 4;
}

// The state-free channelwise weight gradient (backward, and the double backward planned
// without receiver state) writes and reduces its partial rows before the first edge window:
// they share the region of the per-edge contributions.
bool partials_share_contrib(const Plan& p, const WsPlan& w, int pass) {
  const bool free = p.mode == SOBEK_MODE_UVU && p.uvu_C > 0 && p.uvu_bwd_direct && p.uvu_wgrad_direct;
  return free && (pass == SOBEK_PASS_BWD || (pass == SOBEK_PASS_DBWD && w.nstate == 0));
}

size_t layout_total(const Plan& p, WsPlan& w, int pass) {
  size_t o = w.fixed;
  const bool share = partials_share_contrib(p, w, pass);
  const size_t pbytes = pass != SOBEK_PASS_FWD ? partial_floats(p, w.ncap, pass, w.nstate) * 4 : 0;
  if (!share) o = align_up(o + pbytes);
  w.off_K = o;  // w.kfloats is set by the planner
  o = align_up(o + w.kfloats * 4);
  w.off_state = o;
  o = align_up(o + (size_t)w.nstate * w.ncap * p.srow * 4);
  w.off_contrib = o;
  w.off_P = share ? o : w.fixed;
  size_t cbytes = pass != SOBEK_PASS_FWD ? (size_t)w.ecap * (p.dim_in + uvu_edge_partials(p, pass)) * 4 : 0;
  if (share) cbytes = std::max(cbytes, pbytes);
  return align_up(o + cbytes);
}

// nstate: receiver-state slots per receiver (-1: the pass's general need; the
// forward with a retained state needs none, the double backward without dA one)
int plan_workspace(const Plan& p, const sobek_graph_s& G, int pass, size_t ws_bytes, WsPlan& w, bool sizing_only,
                   int nstate = -1) {
  size_t per_recv, per_edge;
  pass_costs(p, G, pass, nstate, w, per_recv, per_edge);
  const int64_t N = G.N, E = G.E;
  // The state-GEMM split-K region only adds blocks: give it what the budget leaves
  // once the chunk capacities are fixed, down to nothing (no split).
  auto fit_split = [&]() -> size_t {
    w.kfloats = sa_split_floats(p, pass, w.ncap);
    size_t t = layout_total(p, w, pass);
    if (t <= ws_bytes || !w.kfloats) return t;
    w.kfloats = 0;
    const size_t bare = layout_total(p, w, pass);
    if (bare >= ws_bytes) return bare;
    w.kfloats = std::min(sa_split_floats(p, pass, w.ncap), (ws_bytes - bare) / kAlign * kAlign / 4);
    return layout_total(p, w, pass);
  };
  // try a single chunk, else split the remaining bytes between state and contributions
  w.ncap = std::max<int64_t>(1, N);
  w.ecap = std::max<int64_t>(G.max_deg, E);
  w.kfloats = 0;
  size_t need = layout_total(p, w, pass);
  if (need <= ws_bytes) {
    need = fit_split();
    w.total = need;
  } else {
    // GEMM partials (weight-gradient splits, state-GEMM split-K) of chunks of nc receivers
    auto partial_bytes = [&](int64_t nc) -> size_t {
      nc = std::max<int64_t>(1, nc);
      return (pass != SOBEK_PASS_FWD ? align_up(partial_floats(p, nc, pass, w.nstate) * 4) + kAlign : 0) +
             align_up(sa_split_floats(p, pass, nc) * 4) + kAlign;
    };
    auto total_at = [&](int64_t nc, int64_t ec, size_t kf) {
      w.ncap = nc;
      w.ecap = ec;
      w.kfloats = kf;
      return layout_total(p, w, pass);
    };
    const int64_t eall = std::max<int64_t>(G.max_deg, E);
    const int64_t ec0 = per_edge ? 1 : eall;
    // A capacity nc of receivers leaves, after the fixed part, the partials, the state of nc
    // receivers and the split-K region (what fits of it), every byte to the per-edge
    // contributions, whose windows of ec edges need not follow receiver boundaries.  Among
    // candidate capacities keep the cheapest, counting a receiver chunk (state, GEMMs, the
    // per-group launches) as four edge windows (one edge kernel and one sender reduction),
    // ties to the larger nc.
    // The split-K region is reserved whole (strict) unless no capacity fits with it.
    struct Cand { int64_t nc = 0, ec = 0; size_t kf = 0, need = 0, score = 0; };
    bool strict = true;
    auto eval = [&](int64_t nc) {
      Cand c;
      c.nc = nc;
      if (strict) {
        c.kf = sa_split_floats(p, pass, nc);
        c.need = total_at(nc, ec0, c.kf);
        if (c.need > ws_bytes) return c;  // infeasible: score 0
      } else {
        if (total_at(nc, ec0, 0) > ws_bytes) return c;
        w.ncap = nc;
        w.ecap = ec0;
        c.need = fit_split();
        c.kf = w.kfloats;
      }
      c.ec = ec0;
      if (per_edge && partials_share_contrib(p, w, pass)) {
        // the largest window that fits (the shared region is not additive in ec)
        int64_t lo = ec0, hi = eall;
        if (total_at(nc, hi, c.kf) <= ws_bytes) lo = hi;
        while (hi - lo > 1) {
          const int64_t mid = lo + (hi - lo) / 2;
          (total_at(nc, mid, c.kf) <= ws_bytes ? lo : hi) = mid;
        }
        c.ec = lo;
        c.need = total_at(nc, lo, c.kf);
      } else if (per_edge) {
        int64_t ec = std::min<int64_t>(eall, ec0 + (int64_t)((ws_bytes - c.need) / per_edge));
        while (ec > ec0 && total_at(nc, ec, c.kf) > ws_bytes) ec = std::max<int64_t>(ec0, ec - 64);
        c.ec = ec;
        c.need = total_at(nc, ec, c.kf);
      }
      const int64_t R = cdiv(N, nc), per_chunk = (std::max<int64_t>(1, E) + R - 1) / R;
      c.score = 4 * (size_t)R + (per_edge ? (size_t)R * cdiv(per_chunk, c.ec) : 0);
      return c;
    };
    std::vector<int64_t> cands;
    for (int64_t nc = std::max<int64_t>(1, N); nc >= 1; nc /= 2) cands.push_back(nc);
    if (per_recv) {
      // the bytes left after the fixed part and the partials, split between receiver state and
      // contributions in proportion to their totals (a few rounds: the partials shrink with nc)
      const double wr = (double)N * per_recv, we = (double)E * per_edge;
      int64_t nc = std::max<int64_t>(1, N);
      for (int iter = 0; iter < 4; ++iter) {
        const size_t aux = partial_bytes(nc);
        if (ws_bytes <= w.fixed + aux) break;
        const double rem = (double)(ws_bytes - w.fixed - aux);
        nc = std::min<int64_t>(std::max<int64_t>(1, (int64_t)(rem * (wr / (wr + we)) / per_recv)), N);
        cands.push_back(nc);
      }
    }
    Cand best;
    for (int pass_strict = 1; pass_strict >= 0 && !best.score; --pass_strict) {
      strict = pass_strict;
      for (int64_t nc : cands) {
        Cand c = eval(nc);
        if (c.score && (!best.score || c.score < best.score || (c.score == best.score && c.nc > best.nc))) best = c;
      }
    }
    if (best.score && best.nc < std::max<int64_t>(1, N)) {
      // refine: the largest capacity with no higher cost (bisection above the best)
      int64_t lo = best.nc, hi = std::min<int64_t>(N, 2 * best.nc);
      while (hi - lo > 1) {
        const int64_t mid = lo + (hi - lo) / 2;
        Cand c = eval(mid);
        if (c.score && c.score <= best.score) {
          best = c;
          lo = mid;
        } else {
          hi = mid;
        }
      }
    }
    if (best.score) {
      total_at(best.nc, best.ec, best.kf);
      need = best.need;
    } else {
      need = total_at(1, ec0, 0);  // not even one receiver fits: report the minimum
    }
    // A chunked pass plans from ws_bytes alone: report the whole budget so that a call
    // given exactly the reported bytes reproduces these chunk capacities.
    w.total = std::max(need, ws_bytes);
  }
  if (sizing_only) return SOBEK_OK;
  if (need > ws_bytes)
    return fail(SOBEK_E_WORKSPACE, "workspace of %zu bytes is below the minimum %zu for this pass", ws_bytes, need);
  // receiver chunks of ncap receivers; the edge kernels walk each chunk's edges in
  // windows of ecap edges
  w.chunks.clear();
  for (int64_t r = 0; r < N; r += w.ncap) {
    const int64_t n = std::min<int64_t>(w.ncap, N - r);
    w.chunks.push_back({(int)r, (int)n, (int64_t)G.h_rowptr[r], (int64_t)G.h_rowptr[r + n]});
  }
  return SOBEK_OK;
}

size_t default_budget() { return (size_t)1 << 30; }

struct Ctx {
  const Plan& p;
  const sobek_graph_s& G;
  hipStream_t s;
};

int fill_zero(const Plan& p, float* buf, int64_t n, hipStream_t s) {
  if (!buf || n <= 0) return SOBEK_OK;
  long long nn = n;
  LAUNCH(p.k.zero, cdiv(n, 256), 1, 1, s, buf, nn);
  return SOBEK_OK;
}

int transpose(const Plan& p, const float* src, float* dst, int64_t N, bool input_side, int dir, hipStream_t s) {
  const int CX = input_side ? p.dim_in : p.dim_out;
  const int nb = input_side ? (int)p.in.size() : (int)p.out.size();
  const int32_t* base = input_side ? p.d_in_blocks : p.d_out_blocks;
  int n = (int)N;
  LAUNCH(p.k.transpose, cdiv(N * CX, 256), 1, 1, s, src, dst, n, CX, (const int*)base, (const int*)(base + nb),
         (const int*)(base + 2 * nb), nb, dir);
  return SOBEK_OK;
}

int zero_dead_out(const Plan& p, float* out, int64_t N, hipStream_t s) {
  for (int c : p.dead_out) {
    int n = (int)N, CX = p.dim_out, off = p.out[c].off, width = p.out[c].dim();
    LAUNCH(p.k.fill_cols, cdiv(N * width, 256), 1, 1, s, out, n, CX, off, width);
  }
  return SOBEK_OK;
}

float* state_ptr(const WsPlan& w, void* ws, const Plan& p, int which) {
  return (float*)((char*)ws + w.off_state) + (size_t)which * w.ncap * p.srow;
}

// Bytes per element of the receiver state S (and dS): bf16 for plans whose channel GEMMs run on
// bf16 MFMA (they round S to bf16 as they read it, so storing it rounded changes nothing but the
// bytes), fp32 otherwise.  The adjoint state S-bar is fp32 for every plan.
size_t state_elem(const Plan& p) { return p.dtype == SOBEK_DTYPE_BF16_GEMM ? 2 : 4; }

// Pointer `elems` state elements past S.
const float* state_at(const Plan& p, const float* S, size_t elems) {
  return (const float*)((const char*)S + elems * state_elem(p));
}

// S (or dS) for the chunk
int run_state(const Plan& p, const sobek_graph_s& G, const Chunk& c, const WsPlan& w, float* S, bool tangent,
              const float* x, const float* evec, const float* phi, const float* xdot, const float* evdot,
              const float* phidot, int flags, hipStream_t s) {
  const int NU = (int)p.fwd_units.size();
  long long ncap = w.ncap;
  int r0 = c.r0, n = c.n;
  hipFunction_t f = !tangent ? p.k.fwd_S : (flags == 4 ? p.k.fwd_dS_r : p.k.fwd_dS);
  LAUNCH(f, cdiv((int64_t)n * NU, 4), 1, 1, s, (const int*)G.rowptr,
         (const int*)G.sender, evec, phi, x, S, r0, n, ncap, xdot, evdot, phidot, flags);
  return SOBEK_OK;
}

// S_g (or dS_g) of output group gi for receivers [r0, r0 + n), written at the start of Sg
// (receiver r0 + il at rows il * d_g ...)
int group_state(const Plan& p, const sobek_graph_s& G, int gi, int r0, int n, float* Sg, bool tangent,
                const float* x, const float* evec, const float* phi, const float* xdot, const float* evdot,
                const float* phidot, int flags, hipStream_t s) {
  const int NU = p.grp_units[gi];
  long long ncap = n;
  hipFunction_t f = p.k.fwd_grp[gi][!tangent ? 0 : (flags == 4 ? 1 : 2)];
  LAUNCH(f, cdiv((int64_t)n * NU, 4), 1, 1, s, (const int*)G.rowptr, (const int*)G.sender, evec, phi, x, Sg, r0, n,
         ncap, xdot, evdot, phidot, flags);
  return SOBEK_OK;
}

// Receivers per chunk of output group g when its state and output rows share `bytes` of fp32
// scratch (Appendix B.2, eq. receiver_chunk_budget: B / (4 d_g (D_g + C_g)), at least one, at most N).
// The state alone, n_g d_g D_g elements of at most 4 bytes, then fits those bytes for any n_g >= 1
// once one receiver's whole state does.
int64_t group_chunk(const sobek::Group& g, int64_t N, size_t bytes) {
  const size_t per = (size_t)4 * g.d * ((size_t)g.D + (size_t)g.C);
  return std::max<int64_t>(1, std::min<int64_t>(std::max<int64_t>(1, N), (int64_t)(bytes / per)));
}

// Bytes of the receiver-state slots of a planned pass: what the per-group legs have to themselves
// (every slot, since the legs that use two slots run after them).
size_t state_region(const Plan& p, const WsPlan& w) { return (size_t)w.nstate * w.ncap * p.srow * 4; }

// Elements before group gi in a kept state of N receivers holding the groups of `mask`
// (group blocks in group order, group g's block N d_g D_g elements).
size_t kept_offset(const Plan& p, int64_t N, uint64_t mask, int gi) {
  size_t o = 0;
  for (int h = 0; h < gi && h < 64; ++h)
    if (mask >> h & 1) o += (size_t)N * p.groups[h].d * p.groups[h].D;
  return o;
}

bool kept(uint64_t mask, int gi) { return gi < 64 && (mask >> gi & 1); }

// Forward-state waves (receivers x wave units) below which an all-group receiver chunk leaves the
// GPU underfilled: eight waves on each of its 1024 SIMDs.
constexpr int64_t kFillWaves = 8 * 1024;

// SOBEK_POLICY_AUTO: the per-group route when the all-group plan of a pass needs at least three
// receiver chunks (Appendix B.2 takes a chunked route only when it gives at least three chunks) and
// each of them is too small to fill the GPU.  The per-group route walks every edge once per output
// group, so with all-group chunks that already fill the GPU it only adds edge traffic.
bool group_route_pays(const Plan& p, const WsPlan& w) {
  return p.policy == SOBEK_POLICY_AUTO && w.chunks.size() >= 3 &&
         w.ncap * (int64_t)p.fwd_units.size() < kFillWaves;
}

// Whether `mask` keeps every output group (never for a plan with more than 64).
bool keeps_all(const Plan& p, uint64_t mask) {
  const size_t G = p.groups.size();
  return mask && G <= 64 && mask == (G == 64 ? ~(uint64_t)0 : (((uint64_t)1 << G) - 1));
}

// out(i, m_o, w) (+)= S_g A_g for group g; Sg holds the group's rows of receivers [r0, r0 + n)
int mix_group(const Plan& p, const sobek::Group& g, int r0, int n, const WsPlan& w, void* ws, const float* Sg,
              const float* W, float* out, int acc, hipStream_t s) {
  float* K = (float*)((char*)ws + w.off_K);
  int nrows = n * g.d, D = (int)g.D, dg = g.d, Cg = g.C, off = g.off, CX = p.dim_out;
  if (p.mode == SOBEK_MODE_UVU) {
    LAUNCH(p.k.uvu_mix, cdiv((int64_t)nrows * Cg, 256), 1, 1, s, Sg, nrows, D, Cg, W,
           (const int*)(p.d_ktab + g.ktab_off), out, dg, off, CX, r0, acc);
    return SOBEK_OK;
  }
  int bn = state_gemm_bn(p, g);
  if (p.vec4) {
    int kper = D;
    const int ns = sa_nsplit(p, g, nrows, w.kfloats, kper);
    LAUNCH(bn == 128 ? p.k.gemm_sa_vb128 : p.k.gemm_sa_v[bn_index(bn)], cdiv(nrows, 128), cdiv(Cg, bn), ns, s, Sg,
           nrows, D, W,
           (const int*)(p.d_ktab + g.ktab_off), out, dg, Cg, off, CX, r0, acc, K, kper);
    if (ns > 1)
      LAUNCH(p.k.sa_reduce, cdiv((int64_t)nrows * (Cg / 4), 256), 1, 1, s, (const float*)K, ns, nrows, Cg, out, dg,
             off, CX, r0, acc);
  } else {
    LAUNCH(p.k.gemm_sa[bn_index(bn)], cdiv(nrows, 64), cdiv(Cg, bn), 1, s, Sg, nrows, D, W,
           (const int*)(p.d_ktab + g.ktab_off), out, dg, Cg, off, CX, r0, acc);
  }
  return SOBEK_OK;
}

// out(i, m_o, w) (+)= S_g A_g for every group
int run_mix(const Plan& p, const Chunk& c, const WsPlan& w, void* ws, const float* S, const float* W, float* out,
            int acc, hipStream_t s) {
  for (auto& g : p.groups)
    if (int rc = mix_group(p, g, c.r0, c.n, w, ws, state_at(p, S, (size_t)w.ncap * g.s_off), W, out, acc, s))
      return rc;
  return SOBEK_OK;
}

// Sbar_g = mbar_g A_g^T for every group
// Sbar of receivers [c.r0, c.r0 + c.n) at row 0 of each group block, group blocks
// s_ncap receivers apart (the chunk slot, or a state kept for every receiver)
int run_sbar(const Plan& p, const Chunk& c, int64_t s_ncap, const float* M, const float* W, float* Sbar,
             hipStream_t s) {
  for (auto& g : p.groups) {
    float* Sg = Sbar + (size_t)s_ncap * g.s_off;
    int nrows = c.n * g.d, D = (int)g.D, dg = g.d, Cg = g.C, off = g.off, CX = p.dim_out, r0 = c.r0;
    if (p.mode == SOBEK_MODE_UVU)
      LAUNCH(p.k.uvu_sbar, cdiv((int64_t)nrows * D, 256), 1, 1, s, M, nrows, D, Cg, W,
             (const int*)(p.d_ktab + g.ktab_off), Sg, dg, off, CX, r0);
    else if (sobek::sbar_streams(p.vec4, g.C))
    {
      // spread the 64-wide column tiles over blockIdx.y until about kSaTarget blocks run,
      // keeping at least four tiles per block
      const int rows = cdiv(nrows, sobek::sbar_block_rows(p, g.C)), ntile = cdiv(D, 64);
      const int gy = std::max(1, std::min((int)cdiv(kSaTarget, rows), ntile / 4));
      LAUNCH(p.k.gemm_sbar_c.at(g.C), rows, gy, 1, s, M, nrows, D, W, (const int*)(p.d_ktab + g.ktab_off), Sg, dg,
             off, CX, r0);
    }
    else
      LAUNCH(p.k.gemm_sbar[2], cdiv(nrows, 64), cdiv(D, 64), 1, s, M, nrows, D, W,
             (const int*)(p.d_ktab + g.ktab_off), Sg, dg, Cg, off, CX, r0);
  }
  return SOBEK_OK;
}

// Weight-gradient split partials of group gi: a region of nsplit_for(p, g, ncap d_g) * D_g * C_g
// floats per group, the groups' regions in group order (ncap = the pass's receiver capacity).
float* ga_partials(const Plan& p, const WsPlan& w, void* ws, int gi) {
  float* P = (float*)((char*)ws + w.off_P);
  for (int h = 0; h < gi; ++h) {
    const sobek::Group& g = p.groups[h];
    P += (size_t)nsplit_for(p, g, (int64_t)w.ncap * g.d) * g.D * g.C;
  }
  return P;
}

// gW += S_g^T mbar_g over the rows of receivers [r0, r0 + n), deterministic: each call adds its
// rows into fixed split partials (the group's first call overwrites them), and its last call sums
// the splits in fixed order into W's layout.  The split count follows the pass's receiver
// capacity, so every call of a group, whatever its receiver count, uses the same partials.
int ga_group(const Plan& p, int gi, int r0, int n, const WsPlan& w, void* ws, const float* Sg, const float* M,
             float* gW, bool first_chunk, bool last_chunk, hipStream_t s) {
  const sobek::Group& g = p.groups[gi];
  float* P = ga_partials(p, w, ws, gi);
  int nrows = n * g.d, D = (int)g.D, dg = g.d, Cg = g.C, off = g.off, CX = p.dim_out;
  int ns = nsplit_for(p, g, (int64_t)w.ncap * g.d);
  int rps = (int)(((int64_t)cdiv(nrows, ns) + 31) / 32 * 32);
  int bn = gemm_bn(g.C);
  int acc = first_chunk ? 0 : 1;
  if (p.mode == SOBEK_MODE_UVU) {
    // channelwise: one weight per column k of S (P[split][k]); the region holds ns * D * C floats
    LAUNCH(p.k.uvu_ga, cdiv(D, 256), 1, ns, s, Sg, nrows, D, Cg, M, P, dg, off, CX, r0, rps, acc);
    if (last_chunk) {
      int one = 1, ncol = 1;
      LAUNCH(p.k.ga_reduce, cdiv((int64_t)D, 256), 1, 1, s, (const float*)P, ns, D, ncol,
             (const int*)(p.d_ktab + g.ktab_off), gW, one);
    }
    return SOBEK_OK;
  }
  if (p.vec4)
    LAUNCH(p.k.gemm_ga_v[bn_index(bn)], cdiv(D, 128), cdiv(Cg, bn), ns, s, Sg, nrows, D, M, P, dg, Cg, off, CX, r0,
           rps, acc);
  else
    LAUNCH(p.k.gemm_ga[bn_index(bn)], cdiv(D, 64), cdiv(Cg, bn), ns, s, Sg, nrows, D, M, P, dg, Cg, off, CX, r0,
           rps, acc);
  if (last_chunk) {
    int one = 1;
    LAUNCH(p.k.ga_reduce, cdiv((int64_t)D * Cg, 256), 1, 1, s, (const float*)P, ns, D, Cg,
           (const int*)(p.d_ktab + g.ktab_off), gW, one);
  }
  return SOBEK_OK;
}

// gW over every group; S holds the state of receivers [c.r0, c.r0 + c.n) at row 0 of each group
// block, group blocks s_ncap receivers apart (the chunk slot, or a retained full state).
int run_ga(const Plan& p, const Chunk& c, const WsPlan& w, void* ws, const float* S, int64_t s_ncap, const float* M,
           float* gW, bool first_chunk, bool last_chunk, hipStream_t s) {
  for (int gi = 0; gi < (int)p.groups.size(); ++gi)
    if (int rc = ga_group(p, gi, c.r0, c.n, w, ws, state_at(p, S, (size_t)s_ncap * p.groups[gi].s_off), M, gW,
                          first_chunk, last_chunk, s))
      return rc;
  return SOBEK_OK;
}

// out (+)= S A, one output group at a time: kept groups from `keep` (one pass over every
// receiver, written there by the forward when `write_kept`), the others recomputed in chunks of
// group_chunk receivers in the state slot.
int fwd_by_group(const Plan& p, const sobek_graph_s& G, const WsPlan& w, void* ws, uint64_t mask, float* keep,
                 bool write_kept, const float* x, const float* evec, const float* phi, const float* W, float* out,
                 hipStream_t s) {
  int rc;
  float* slot = state_ptr(w, ws, p, 0);
  for (int gi = 0; gi < (int)p.groups.size(); ++gi) {
    const sobek::Group& g = p.groups[gi];
    if (kept(mask, gi)) {
      float* Sg = (float*)state_at(p, keep, kept_offset(p, G.N, mask, gi));
      if (write_kept && (rc = group_state(p, G, gi, 0, (int)G.N, Sg, false, x, evec, phi, nullptr, nullptr, nullptr,
                                          0, s)))
        return rc;
      if ((rc = mix_group(p, g, 0, (int)G.N, w, ws, Sg, W, out, 0, s))) return rc;
      continue;
    }
    const int64_t ng = group_chunk(g, G.N, state_region(p, w));
    for (int64_t r = 0; r < G.N; r += ng) {
      const int n = (int)std::min<int64_t>(ng, G.N - r);
      if ((rc = group_state(p, G, gi, (int)r, n, slot, false, x, evec, phi, nullptr, nullptr, nullptr, 0, s)) ||
          (rc = mix_group(p, g, (int)r, n, w, ws, slot, W, out, 0, s)))
        return rc;
    }
  }
  return SOBEK_OK;
}

// gW = S^T mbar, one output group at a time: kept groups read from `keep` in one pass, the others
// recomputed in chunks of group_chunk receivers in the state slot.
int ga_by_group(const Plan& p, const sobek_graph_s& G, const WsPlan& w, void* ws, uint64_t mask, const float* keep,
                const float* x, const float* evec, const float* phi, const float* M, float* gW, hipStream_t s) {
  int rc;
  float* slot = state_ptr(w, ws, p, 0);
  for (int gi = 0; gi < (int)p.groups.size(); ++gi) {
    if (kept(mask, gi)) {
      if ((rc = ga_group(p, gi, 0, (int)G.N, w, ws, state_at(p, keep, kept_offset(p, G.N, mask, gi)), M, gW, true,
                         true, s)))
        return rc;
      continue;
    }
    const int64_t ng = group_chunk(p.groups[gi], G.N, state_region(p, w));
    for (int64_t r = 0; r < G.N; r += ng) {
      const int n = (int)std::min<int64_t>(ng, G.N - r);
      if ((rc = group_state(p, G, gi, (int)r, n, slot, false, x, evec, phi, nullptr, nullptr, nullptr, 0, s)) ||
          (rc = ga_group(p, gi, (int)r, n, w, ws, slot, M, gW, r == 0, r + n >= G.N, s)))
        return rc;
    }
  }
  return SOBEK_OK;
}

// The double backward's receiver-state legs, one output group at a time in chunks of group_chunk
// receivers: dS_g for the output tangent (ggk) and the weight gradient (g_W), then S_g for the
// output tangent's S dA term (t_gW), in the state slot.
int dbwd_state_by_group(const Plan& p, const sobek_graph_s& G, const WsPlan& w, void* ws, const float* x,
                        const float* evec, const float* phi, const float* xdot, const float* evdot,
                        const float* phidot, int flags, const float* W, const float* t_gW, const float* gk,
                        float* ggk, float* g_W, hipStream_t s) {
  int rc;
  const bool tan = flags & 7;
  float* slot = state_ptr(w, ws, p, 0);
  for (int gi = 0; gi < (int)p.groups.size(); ++gi) {
    const sobek::Group& g = p.groups[gi];
    const int64_t ng = group_chunk(g, G.N, state_region(p, w));
    for (int64_t r = 0; r < G.N; r += ng) {
      const int r0 = (int)r, n = (int)std::min<int64_t>(ng, G.N - r);
      if (tan && (ggk || g_W)) {
        if ((rc = group_state(p, G, gi, r0, n, slot, true, x, evec, phi, xdot, evdot, phidot, flags & 7, s))) return rc;
        if (ggk && (rc = mix_group(p, g, r0, n, w, ws, slot, W, ggk, 0, s))) return rc;
        if (g_W && (rc = ga_group(p, gi, r0, n, w, ws, slot, gk, g_W, r == 0, r + n >= G.N, s))) return rc;
      }
      if (t_gW && ggk) {  // S_g reuses the slot once dS_g has been consumed
        if ((rc = group_state(p, G, gi, r0, n, slot, false, x, evec, phi, nullptr, nullptr, nullptr, 0, s)) ||
            (rc = mix_group(p, g, r0, n, w, ws, slot, t_gW, ggk, tan ? 1 : 0, s)))
          return rc;
      }
    }
  }
  return SOBEK_OK;
}

int run_sender_reduce(const Plan& p, const sobek_graph_s& G, int64_t ea, int64_t eb, const WsPlan& w, void* ws,
                      const float* contrib, float* gx, int first, hipStream_t s) {
  int N = (int)G.N, CX = p.dim_in, e0 = (int)ea, e1 = (int)eb;
  int* cursor = (int*)((char*)ws + w.off_cursor);
  LAUNCH(p.k.sender_reduce, cdiv(G.N, 4), 1, 1, s, (const int*)G.send_rowptr, (const int*)G.send_perm, contrib, gx,
         cursor, N, CX, e0, e1, first);
  return SOBEK_OK;
}

// Edge windows of a receiver chunk for the edge-owned adjoint kernels: consecutive
// ranges of at most w.ecap edges (the x-gradient contribution buffer), each handed
// to f(ea, eb, ra, nr) with the receivers [ra, ra + nr) that own its edges.
template <class F>
int for_edge_windows(const sobek_graph_s& G, const Chunk& c, const WsPlan& w, F&& f) {
  const int32_t* rp = G.h_rowptr.data();
  // equal windows: the fewest that respect the capacity
  const int64_t ne = c.e1 - c.e0, cap = std::max<int64_t>(1, w.ecap);
  const int64_t step = ne > 0 ? (ne + (ne + cap - 1) / cap - 1) / ((ne + cap - 1) / cap) : 1;
  for (int64_t ea = c.e0; ea < c.e1; ea += step) {
    const int64_t eb = std::min<int64_t>(c.e1, ea + step);
    const int ra = (int)(std::upper_bound(rp + c.r0, rp + c.r0 + c.n + 1, (int32_t)ea) - rp) - 1;
    const int rb = (int)(std::lower_bound(rp + c.r0, rp + c.r0 + c.n + 1, (int32_t)eb) - rp);
    if (int rc = f(ea, eb, ra, rb - ra)) return rc;
  }
  return SOBEK_OK;
}

// blockIdx.y split of the adjoint edge kernels: spread the window's receivers' edges
// until about 512 blocks run, at least one 16-edge batch per block (with few receivers a
// block's staged slabs are latency-bound, so shorter edge shares run in parallel)
int adj_edge_split(const Plan& p, int nr, int64_t ne) {
  (void)p;
  const int64_t per_block = 16;
  const int64_t by_work = std::max<int64_t>(1, (ne / std::max(1, nr) + per_block - 1) / per_block);
  return (int)std::max<int64_t>(1, std::min<int64_t>({cdiv(512, std::max(1, nr)), by_work, 64}));
}

int check_common(sobek_plan plan, sobek_graph graph, const float* x, const float* evec, const float* phi,
                 const float* W, void* ws, size_t ws_bytes) {
  if (!plan || !graph) return fail(SOBEK_E_INVALID, "NULL plan or graph");
  if (graph->N > 0 && !x) return fail(SOBEK_E_INVALID, "x is NULL");
  if (graph->E > 0 && (!evec || !phi)) return fail(SOBEK_E_INVALID, "evec or phi is NULL");
  if (!W) return fail(SOBEK_E_INVALID, "W is NULL");
  if (!ws && ws_bytes) return fail(SOBEK_E_WORKSPACE, "workspace pointer is NULL");
  for (const void* q : {(const void*)x, (const void*)evec, (const void*)phi, (const void*)W, (const void*)ws})
    if (q && !aligned16(q)) return fail(SOBEK_E_ALIGN, "pointer %p is not 16-byte aligned", q);
  if (graph->N >= (1ll << 31) || graph->E >= (1ll << 31)) return fail(SOBEK_E_UNSUPPORTED, "graph too large");
  if (graph->N * (int64_t)std::max(plan->p.dim_in, plan->p.dim_out) >= (1ll << 31) * 64ll)
    return fail(SOBEK_E_UNSUPPORTED, "feature tensor too large");
  return SOBEK_OK;
}

}  // namespace

// ============================================================================
extern "C" {

const char* sobek_last_error(void) { return g_err.c_str(); }
int sobek_version(void) { return 1; }

}  // extern "C"

namespace {

int load_module(const std::string& src, hipModule_t& m) {
  std::vector<char> code;
  try {
    code = sobek::jit_compile(src);
  } catch (const std::exception& ex) {
    return fail(SOBEK_E_COMPILE, "%s", ex.what());
  }
  HIPCHK(hipModuleLoadData(&m, code.data()));
  return SOBEK_OK;
}

int get_fn(hipModule_t m, hipFunction_t& f, const char* name) {
  hipError_t e = hipModuleGetFunction(&f, m, name);
  if (e != hipSuccess) return fail(SOBEK_E_INTERNAL, "kernel %s missing: %s", name, hipGetErrorString(e));
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_names[f] = name;
  return SOBEK_OK;
}

// kernels every route uses (prelude and the sender gather)
int load_common(Plan& p, hipModule_t m) {
  int rc;
  if ((rc = get_fn(m, p.k.ga_reduce, "sobek_ga_reduce")) || (rc = get_fn(m, p.k.sender_reduce, "sobek_sender_reduce")) ||
      (rc = get_fn(m, p.k.transpose, "sobek_transpose")) || (rc = get_fn(m, p.k.fill_cols, "sobek_fill_cols")) ||
      (rc = get_fn(m, p.k.zero, "sobek_zero")) || (rc = get_fn(m, p.k.sa_reduce, "sobek_sa_reduce")) ||
      (rc = get_fn(m, p.k.uvu_mix, "sobek_uvu_mix")) || (rc = get_fn(m, p.k.uvu_sbar, "sobek_uvu_sbar")) ||
      (rc = get_fn(m, p.k.uvu_ga, "sobek_uvu_ga")))
    return rc;
  return SOBEK_OK;
}

// the receiver-state route: state and adjoint edge kernels, channel GEMMs
int load_receiver_route(Plan& p, hipModule_t m) {
  int rc;
  if ((rc = get_fn(m, p.k.fwd_S, "sobek_fwd_S")) || (rc = get_fn(m, p.k.fwd_dS, "sobek_fwd_dS")) ||
      (rc = get_fn(m, p.k.fwd_dS_r, "sobek_fwd_dS_r")) || (rc = get_fn(m, p.k.bwd_E, "sobek_bwd_E")) ||
      (rc = get_fn(m, p.k.dbwd_E, "sobek_dbwd_E")) || (rc = get_fn(m, p.k.dbwd_E_r, "sobek_dbwd_E_r")))
    return rc;
  const char* bns[3] = {"16", "32", "64"};
  for (int b = 0; b < 3; ++b) {
    std::string sa = std::string("sobek_gemm_sa_") + bns[b], sb = std::string("sobek_gemm_sbar_") + bns[b],
                ga = std::string("sobek_gemm_ga_") + bns[b],
                sav = std::string(p.dtype == SOBEK_DTYPE_BF16_GEMM ? "sobek_gemm_sa_vb" : "sobek_gemm_sa_v") + bns[b],
                gav = std::string(p.dtype == SOBEK_DTYPE_BF16_GEMM ? "sobek_gemm_ga_vb" : "sobek_gemm_ga_v") + bns[b];
    if ((rc = get_fn(m, p.k.gemm_sa[b], sa.c_str())) || (rc = get_fn(m, p.k.gemm_sbar[b], sb.c_str())) ||
        (rc = get_fn(m, p.k.gemm_ga[b], ga.c_str())) || (rc = get_fn(m, p.k.gemm_sa_v[b], sav.c_str())) ||
        (rc = get_fn(m, p.k.gemm_ga_v[b], gav.c_str())))
      return rc;
  }
  if ((rc = get_fn(m, p.k.gemm_sbar_v, "sobek_gemm_sbar_v"))) return rc;
  if (p.dtype == SOBEK_DTYPE_BF16_GEMM && (rc = get_fn(m, p.k.gemm_sa_vb128, "sobek_gemm_sa_vb128"))) return rc;
  if (p.vec4)
    for (auto& g : p.groups)
      if (sobek::sbar_streams(p.vec4, g.C) && !p.k.gemm_sbar_c.count(g.C)) {
        std::string nm = (sobek::sbar_bf16(p, g.C) ? "sobek_gemm_sbar_cb" : "sobek_gemm_sbar_c") + std::to_string(g.C);
        hipFunction_t f = nullptr;
        if ((rc = get_fn(m, f, nm.c_str()))) return rc;
        p.k.gemm_sbar_c[g.C] = f;
      }
  return SOBEK_OK;
}

// channelwise state-free kernels, with the route choice from their scratch and register use
int load_uvu(Plan& p, hipModule_t m) {
  int rc;
  auto get = [&](hipFunction_t& f, const char* name) { return get_fn(m, f, name); };
  hipFunction_t bu = nullptr, bs = nullptr;
  if ((rc = get(p.k.uvu_fwd, "sobek_uvu_fwd")) || (rc = get(bu, "sobek_uvu_bwd_u")) ||
      (rc = get(bs, "sobek_uvu_bwd_s")))
    return rc;
  if ((rc = get(p.k.uvu_wgrad, "sobek_uvu_wgrad")) || (rc = get(p.k.uvu_wreduce, "sobek_uvu_wreduce"))) return rc;
  // many paths at high order make the state-free backward spill registers to scratch,
  // which is slower than the receiver route: take the all-irrep form when it compiled
  // without spills and below the 256-register cap (two waves per SIMD), else the
  // per-input-irrep form, else the receiver route
  int su = 0, ss = 0, sw = 0, ru = 0;
  HIPCHK(hipFuncGetAttribute(&su, HIP_FUNC_ATTRIBUTE_LOCAL_SIZE_BYTES, bu));
  HIPCHK(hipFuncGetAttribute(&ss, HIP_FUNC_ATTRIBUTE_LOCAL_SIZE_BYTES, bs));
  HIPCHK(hipFuncGetAttribute(&sw, HIP_FUNC_ATTRIBUTE_LOCAL_SIZE_BYTES, p.k.uvu_wgrad));
  HIPCHK(hipFuncGetAttribute(&ru, HIP_FUNC_ATTRIBUTE_NUM_REGS, bu));
  p.uvu_bwd_direct = su == 0 || ss == 0;
  p.uvu_sliced = su != 0 || (ru >= 256 && ss == 0);
  // SOBEK_UVU_FORM=u|s forces one form (testing: both forms run on any signature; a form that
  // spills is slower, not wrong)
  const char* form = std::getenv("SOBEK_UVU_FORM");
  const bool forced = form && (std::strcmp(form, "u") == 0 || std::strcmp(form, "s") == 0);
  if (forced) {
    p.uvu_bwd_direct = true;
    p.uvu_sliced = form[0] == 's';
  }
  p.k.uvu_bwd = p.uvu_sliced ? bs : bu;
  const int npart = p.uvu_NB * (p.uvu_sliced ? p.uvu_NA : 1);
  if (p.uvu_bwd_direct && npart > 1 &&
      (rc = get(p.k.uvu_bwd_fin, p.uvu_sliced ? "sobek_uvu_bwd_fin_s" : "sobek_uvu_bwd_fin_u")))
    return rc;
  p.uvu_wgrad_direct = sw == 0;
  // the edge-vector-tangent variants (double backward), same slicing
  if ((rc = get(p.k.uvu_fwd_t, "sobek_uvu_fwd_t")) || (rc = get(p.k.uvu_wgrad_t, "sobek_uvu_wgrad_t")) ||
      (rc = get(p.k.uvu_bwd_t, p.uvu_sliced ? "sobek_uvu_bwd_st" : "sobek_uvu_bwd_ut")))
    return rc;
  if (p.uvu_bwd_direct && npart > 1 &&
      (rc = get(p.k.uvu_bwd_fin_t, p.uvu_sliced ? "sobek_uvu_bwd_fin_st" : "sobek_uvu_bwd_fin_ut")))
    return rc;
  int st = 0, swt = 0;
  HIPCHK(hipFuncGetAttribute(&st, HIP_FUNC_ATTRIBUTE_LOCAL_SIZE_BYTES, p.k.uvu_bwd_t));
  HIPCHK(hipFuncGetAttribute(&swt, HIP_FUNC_ATTRIBUTE_LOCAL_SIZE_BYTES, p.k.uvu_wgrad_t));
  p.uvu_tan_direct = (st == 0 || forced) && swt == 0;
  return SOBEK_OK;
}

std::mutex g_rr_mu;

// the receiver-route kernels of a channelwise plan, compiled and loaded on first use
// The materialized baseline covers fully connected plans in the ir_mul layout with fp32 GEMMs.
bool materialized_supported(const Plan& p) {
  return p.mode == SOBEK_MODE_UVW && p.layout == SOBEK_LAYOUT_IR_MUL && p.dtype == SOBEK_DTYPE_F32;
}

std::mutex g_mat_mu;

int ensure_materialized(sobek_plan plan) {
  Plan& p = plan->p;
  std::lock_guard<std::mutex> lk(g_mat_mu);
  if (p.k.module_mat) return SOBEK_OK;
  hipModule_t m = nullptr;
  int rc;
  if ((rc = load_module(sobek::generate_materialized_source(p), m))) return rc;
  if ((rc = get_fn(m, p.k.mat_w, "sobek_mat_w")) || (rc = get_fn(m, p.k.mat_msg, "sobek_mat_msg")) ||
      (rc = get_fn(m, p.k.mat_reduce, "sobek_mat_reduce"))) {
    (void)hipModuleUnload(m);
    return rc;
  }
  p.k.module_mat = m;
  return SOBEK_OK;
}

// Bytes per edge of the materialized forward's workspace: W (N_w floats) and M (C_out floats).
size_t materialized_edge_bytes(const Plan& p) { return ((size_t)p.n_w + (size_t)p.dim_out) * 4; }

// Edges per W-kernel block (its grid's second axis counts blocks of them).
constexpr int64_t kMatEdgeTile = 32;
constexpr int64_t kMatMaxWindow = 65535 * kMatEdgeTile;

int ensure_receiver_route(sobek_plan plan) {
  Plan& p = plan->p;
  std::lock_guard<std::mutex> lk(g_rr_mu);
  if (p.rr_loaded) return SOBEK_OK;
  int rc;
  if ((rc = load_module(p.source, p.k.module))) return rc;
  if ((rc = load_receiver_route(p, p.k.module))) return rc;
  p.rr_loaded = true;
  return SOBEK_OK;
}

std::mutex g_grp_mu;

// The state kernels of one output group at a time (the per-group scratch policy and group
// retention), a module of their own compiled and loaded on first use.
int ensure_groups(sobek_plan plan) {
  Plan& p = plan->p;
  std::lock_guard<std::mutex> lk(g_grp_mu);
  if (p.k.module_grp) return SOBEK_OK;
  hipModule_t m = nullptr;
  int rc;
  if ((rc = load_module(sobek::generate_group_source(p), m))) return rc;
  std::vector<std::array<hipFunction_t, 3>> fns(p.groups.size());
  std::vector<int> units;
  const char* kinds[3] = {"S", "dS_r", "dS"};
  for (int gi = 0; gi < (int)p.groups.size(); ++gi) {
    for (int k = 0; k < 3; ++k) {
      const std::string nm = "sobek_fwdg" + std::to_string(gi) + "_" + kinds[k];
      if ((rc = get_fn(m, fns[gi][k], nm.c_str()))) {
        (void)hipModuleUnload(m);
        return rc;
      }
    }
    units.push_back((int)sobek::pack_fwd_units(p, gi, nullptr).size());
    if (!units.back()) {
      (void)hipModuleUnload(m);
      return fail(SOBEK_E_INTERNAL, "output group %d has no forward units", gi);
    }
  }
  p.grp_units = units;
  p.k.fwd_grp = fns;
  p.k.module_grp = m;
  return SOBEK_OK;
}

}  // namespace

extern "C" {

int sobek_plan_create(const sobek_irrep* in, int n_in, int lmax, const sobek_irrep* out, int n_out, int K, int mode,
                      int layout, int dtype, int path_norm, sobek_plan* plan) {
  if (!plan) return fail(SOBEK_E_INVALID, "plan output pointer is NULL");
  *plan = nullptr;
  std::unique_ptr<sobek_plan_s> h(new sobek_plan_s());
  Plan& p = h->p;
  int rc = build_signature(in, n_in, lmax, out, n_out, K, mode, layout, dtype, path_norm, p);
  if (rc != SOBEK_OK) return rc;
  // channelwise plans with the state-free kernels compile that part first; the
  // receiver-route kernels follow on first use (ensure_receiver_route)
  const bool split = !p.source_u.empty();
  if ((rc = load_module(split ? p.source_u : p.source, split ? p.k.module_u : p.k.module))) return rc;
  hipModule_t m0 = split ? p.k.module_u : p.k.module;
  if ((rc = load_common(p, m0))) return rc;
  if (p.mode == SOBEK_MODE_UVU && p.uvu_C > 0 && (rc = load_uvu(p, m0))) return rc;
  if (!split) {
    if ((rc = load_receiver_route(p, p.k.module))) return rc;
    p.rr_loaded = true;
  }
  HIPCHK(hipMalloc(&p.d_ktab, std::max<size_t>(4, p.ktab.size() * 4)));
  HIPCHK(hipMemcpy(p.d_ktab, p.ktab.data(), p.ktab.size() * 4, hipMemcpyHostToDevice));
  auto blocks = [](const std::vector<sobek::Irrep>& v) {
    std::vector<int32_t> b(3 * v.size());
    for (size_t i = 0; i < v.size(); ++i) {
      b[i] = v[i].off;
      b[v.size() + i] = v[i].mul;
      b[2 * v.size() + i] = 2 * v[i].l + 1;
    }
    return b;
  };
  auto bi = blocks(p.in), bo = blocks(p.out);
  HIPCHK(hipMalloc(&p.d_in_blocks, bi.size() * 4));
  HIPCHK(hipMemcpy(p.d_in_blocks, bi.data(), bi.size() * 4, hipMemcpyHostToDevice));
  HIPCHK(hipMalloc(&p.d_out_blocks, bo.size() * 4));
  HIPCHK(hipMemcpy(p.d_out_blocks, bo.data(), bo.size() * 4, hipMemcpyHostToDevice));
  *plan = h.release();
  return SOBEK_OK;
}

int sobek_jit_compile(const sobek_irrep* in, int n_in, int lmax, const sobek_irrep* out, int n_out, int K, int mode,
                      int layout, int dtype, int path_norm) {
  Plan p;
  int rc = build_signature(in, n_in, lmax, out, n_out, K, mode, layout, dtype, path_norm, p);
  if (rc != SOBEK_OK) return rc;
  try {
    if (!p.source_u.empty()) sobek::jit_compile(p.source_u);
    // SOBEK_JIT_STATE_FREE_ONLY=1: channelwise plans compile only the part a plan loads at creation
    const char* sf = std::getenv("SOBEK_JIT_STATE_FREE_ONLY");
    if (p.source_u.empty() || !sf || std::strcmp(sf, "1") != 0) sobek::jit_compile(p.source);
    if (materialized_supported(p)) sobek::jit_compile(sobek::generate_materialized_source(p));
    const char* gs = std::getenv("SOBEK_JIT_GROUPS");
    if (gs && std::strcmp(gs, "1") == 0) sobek::jit_compile(sobek::generate_group_source(p));
  } catch (const std::exception& ex) {
    return fail(SOBEK_E_COMPILE, "%s", ex.what());
  }
  return SOBEK_OK;
}

int sobek_plan_source(const sobek_irrep* in, int n_in, int lmax, const sobek_irrep* out, int n_out, int K, int mode,
                      int layout, int dtype, int path_norm, char* buf, size_t buf_bytes, size_t* needed) {
  Plan p;
  int rc = build_signature(in, n_in, lmax, out, n_out, K, mode, layout, dtype, path_norm, p);
  if (rc != SOBEK_OK) return rc;
  std::string s = sobek::full_source(p.source);
  if (needed) *needed = s.size() + 1;
  if (buf && buf_bytes) {
    size_t n = std::min(buf_bytes - 1, s.size());
    std::memcpy(buf, s.data(), n);
    buf[n] = 0;
  }
  return SOBEK_OK;
}

int sobek_profile_enable(int on) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_on = on != 0;
  return SOBEK_OK;
}

int sobek_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto& r : g_prof) {
    g_event_pool.push_back(r.a);
    g_event_pool.push_back(r.b);
  }
  g_prof.clear();
  return SOBEK_OK;
}

int sobek_profile_query(int idx, char* name, size_t name_bytes, int64_t* launches, double* total_ms) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  std::map<std::string, std::pair<int64_t, double>> agg;
  for (auto& r : g_prof) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess) return fail(SOBEK_E_HIP, "profile event: %s", hipGetErrorString(e));
    auto& v = agg[r.name];
    v.first += 1;
    v.second += ms;
  }
  if (idx < 0 || idx >= (int)agg.size()) return fail(SOBEK_E_INVALID, "profile index %d out of range", idx);
  auto it = agg.begin();
  std::advance(it, idx);
  if (name && name_bytes) {
    std::snprintf(name, name_bytes, "%s", it->first.c_str());
  }
  if (launches) *launches = it->second.first;
  if (total_ms) *total_ms = it->second.second;
  return SOBEK_OK;
}

int sobek_plan_destroy(sobek_plan plan) {
  if (!plan) return SOBEK_OK;
  Plan& p = plan->p;
  if (p.d_ktab) (void)hipFree(p.d_ktab);
  if (p.d_in_blocks) (void)hipFree(p.d_in_blocks);
  if (p.d_out_blocks) (void)hipFree(p.d_out_blocks);
  if (p.k.module) (void)hipModuleUnload(p.k.module);
  if (p.k.module_u) (void)hipModuleUnload(p.k.module_u);
  if (p.k.module_mat) (void)hipModuleUnload(p.k.module_mat);
  if (p.k.module_grp) (void)hipModuleUnload(p.k.module_grp);
  if (plan->side) (void)hipStreamDestroy(plan->side);
  if (plan->fork) (void)hipEventDestroy(plan->fork);
  if (plan->join) (void)hipEventDestroy(plan->join);
  delete plan;
  return SOBEK_OK;
}

int sobek_plan_info(sobek_plan plan, int64_t* n_paths, int64_t* n_weights, int64_t* dim_in, int64_t* dim_out,
                    int64_t* dim_sh) {
  if (!plan) return fail(SOBEK_E_INVALID, "NULL plan");
  const Plan& p = plan->p;
  if (n_paths) *n_paths = (int64_t)p.paths.size();
  if (n_weights) *n_weights = p.n_w;
  if (dim_in) *dim_in = p.dim_in;
  if (dim_out) *dim_out = p.dim_out;
  if (dim_sh) *dim_sh = p.nsh;
  return SOBEK_OK;
}

int sobek_plan_paths(sobek_plan plan, int32_t* i_in, int32_t* i_sh, int32_t* i_out, int64_t* w_offset) {
  if (!plan) return fail(SOBEK_E_INVALID, "NULL plan");
  const Plan& p = plan->p;
  for (size_t t = 0; t < p.paths.size(); ++t) {
    if (i_in) i_in[t] = p.paths[t].i_in;
    if (i_sh) i_sh[t] = p.paths[t].i_sh;
    if (i_out) i_out[t] = p.paths[t].i_out;
    if (w_offset) w_offset[t] = p.paths[t].w_off;
  }
  return SOBEK_OK;
}

int sobek_plan_cg(sobek_plan plan, int path, double* coeff) {
  if (!plan || !coeff) return fail(SOBEK_E_INVALID, "NULL argument");
  const Plan& p = plan->p;
  if (path < 0 || path >= (int)p.paths.size()) return fail(SOBEK_E_INVALID, "path index out of range");
  const auto& c = p.paths[path].cg;
  std::copy(c.begin(), c.end(), coeff);
  return SOBEK_OK;
}

int sobek_cg_table(int l1, int l2, int l3, double* coeff) {
  if (!coeff) return fail(SOBEK_E_INVALID, "NULL coeff");
  if (l1 < 0 || l2 < 0 || l3 < 0 || l1 > 8 || l2 > 8 || l3 > 8) return fail(SOBEK_E_INVALID, "bad orders");
  if (l3 < std::abs(l1 - l2) || l3 > l1 + l2) return fail(SOBEK_E_INVALID, "triangle rule violated");
  const auto& Q = sobek::real_cg(l1, l2, l3);
  std::copy(Q.begin(), Q.end(), coeff);
  return SOBEK_OK;
}

int sobek_sh_table(int l, int m, int32_t* n_terms, double* coeff, int32_t* powers, int max_terms) {
  if (l < 0 || l > 8 || m < -l || m > l) return fail(SOBEK_E_INVALID, "bad (l, m)");
  const auto& P = sobek::sh_poly(l, m);
  if (n_terms) *n_terms = (int32_t)P.size();
  for (int t = 0; t < (int)P.size() && t < max_terms; ++t) {
    if (coeff) coeff[t] = P[t].c;
    if (powers) {
      powers[3 * t] = P[t].px;
      powers[3 * t + 1] = P[t].py;
      powers[3 * t + 2] = P[t].pz;
    }
  }
  return SOBEK_OK;
}

int sobek_graph_prepare_size(int64_t N, int64_t E, size_t* bytes) {
  if (!bytes) return fail(SOBEK_E_INVALID, "NULL bytes");
  if (N < 0 || E < 0) return fail(SOBEK_E_INVALID, "negative size");
  *bytes = align_up((size_t)(N + 1) * 4) + align_up((size_t)std::max<int64_t>(E, 1) * 4);
  return SOBEK_OK;
}

int sobek_graph_prepare(const int32_t* recv_rowptr, const int32_t* sender, int64_t N, int64_t E, void* buf,
                        size_t bytes, sobek_graph* graph, hipStream_t stream) {
  if (!graph) return fail(SOBEK_E_INVALID, "graph output pointer is NULL");
  *graph = nullptr;
  if (N < 0 || E < 0) return fail(SOBEK_E_INVALID, "negative size");
  if (N >= (1ll << 31) || E >= (1ll << 31)) return fail(SOBEK_E_UNSUPPORTED, "graph too large for int32 indices");
  if (!recv_rowptr || (E > 0 && !sender)) return fail(SOBEK_E_INVALID, "NULL CSR array");
  size_t need;
  sobek_graph_prepare_size(N, E, &need);
  if (!buf || bytes < need) return fail(SOBEK_E_WORKSPACE, "graph buffer needs %zu bytes", need);
  if (!aligned16(buf)) return fail(SOBEK_E_ALIGN, "graph buffer is not 16-byte aligned");
  std::unique_ptr<sobek_graph_s> g(new sobek_graph_s());
  g->N = N; g->E = E; g->rowptr = recv_rowptr; g->sender = sender;
  g->h_rowptr.resize(N + 1);
  std::vector<int32_t> hs(E);
  HIPCHK(hipMemcpyAsync(g->h_rowptr.data(), recv_rowptr, (N + 1) * 4, hipMemcpyDeviceToHost, stream));
  if (E) HIPCHK(hipMemcpyAsync(hs.data(), sender, E * 4, hipMemcpyDeviceToHost, stream));
  HIPCHK(hipStreamSynchronize(stream));
  if (g->h_rowptr[0] != 0 || g->h_rowptr[N] != E) return fail(SOBEK_E_INVALID, "rowptr must start at 0 and end at E");
  for (int64_t i = 0; i < N; ++i) {
    int64_t d = (int64_t)g->h_rowptr[i + 1] - g->h_rowptr[i];
    if (d < 0) return fail(SOBEK_E_INVALID, "rowptr decreases at %lld", (long long)i);
    g->max_deg = std::max(g->max_deg, d);
  }
  // stable counting sort by sender: inside one sender, edges keep receiver order
  std::vector<int32_t> srow(N + 1, 0), perm(E);
  for (int64_t e = 0; e < E; ++e) {
    if (hs[e] < 0 || hs[e] >= N) return fail(SOBEK_E_INVALID, "sender[%lld] = %d out of range", (long long)e, hs[e]);
    srow[hs[e] + 1]++;
  }
  for (int64_t i = 0; i < N; ++i) srow[i + 1] += srow[i];
  std::vector<int32_t> pos(srow.begin(), srow.end() - 1);
  for (int64_t e = 0; e < E; ++e) perm[pos[hs[e]]++] = (int32_t)e;
  g->send_rowptr = (int32_t*)buf;
  g->send_perm = (int32_t*)((char*)buf + align_up((size_t)(N + 1) * 4));
  HIPCHK(hipMemcpyAsync(g->send_rowptr, srow.data(), (N + 1) * 4, hipMemcpyHostToDevice, stream));
  if (E) HIPCHK(hipMemcpyAsync(g->send_perm, perm.data(), E * 4, hipMemcpyHostToDevice, stream));
  HIPCHK(hipStreamSynchronize(stream));
  *graph = g.release();
  return SOBEK_OK;
}

int sobek_graph_destroy(sobek_graph graph) {
  delete graph;
  return SOBEK_OK;
}

int sobek_graph_info(sobek_graph graph, int64_t* N, int64_t* E) {
  if (!graph) return fail(SOBEK_E_INVALID, "NULL graph");
  if (N) *N = graph->N;
  if (E) *E = graph->E;
  return SOBEK_OK;
}

int sobek_workspace_size(sobek_plan plan, sobek_graph graph, int pass, size_t budget, size_t* bytes) {
  if (!plan || !graph || !bytes) return fail(SOBEK_E_INVALID, "NULL argument");
  if (pass < SOBEK_PASS_FWD || pass > SOBEK_PASS_DBWD) return fail(SOBEK_E_INVALID, "bad pass");
  WsPlan w;
  const size_t b = budget ? budget : default_budget();
  plan_workspace(plan->p, *graph, pass, b, w, true);
  *bytes = w.total;
  // a channelwise double backward may take the state-free route (edge-vector cotangent
  // alone): room for its layout too
  const Plan& p = plan->p;
  if (pass == SOBEK_PASS_DBWD && p.mode == SOBEK_MODE_UVU && p.uvu_C > 0 && p.uvu_bwd_direct &&
      p.uvu_wgrad_direct) {
    WsPlan w0;
    plan_workspace(p, *graph, pass, b, w0, true, 0);
    *bytes = std::max(*bytes, w0.total);
  }
  return SOBEK_OK;
}

}  // extern "C"

namespace {

// Fork: work queued on the returned side stream after this call runs after everything queued on
// `main` so far.  The side stream is the plan's own; calls on one plan serialise their side work.
int side_fork(sobek_plan plan, hipStream_t main, hipStream_t& side) {
  std::lock_guard<std::mutex> lk(plan->side_mu);
  if (!plan->side) {
    HIPCHK(hipStreamCreateWithFlags(&plan->side, hipStreamNonBlocking));
    HIPCHK(hipEventCreateWithFlags(&plan->fork, hipEventDisableTiming));
    HIPCHK(hipEventCreateWithFlags(&plan->join, hipEventDisableTiming));
  }
  HIPCHK(hipEventRecord(plan->fork, main));
  HIPCHK(hipStreamWaitEvent(plan->side, plan->fork, 0));
  side = plan->side;
  return SOBEK_OK;
}

// Join: work queued on `main` after this call runs after everything queued on the side stream so far.
int side_join(sobek_plan plan, hipStream_t main) {
  std::lock_guard<std::mutex> lk(plan->side_mu);
  HIPCHK(hipEventRecord(plan->join, plan->side));
  HIPCHK(hipStreamWaitEvent(main, plan->join, 0));
  return SOBEK_OK;
}

// Forward; with `state` non-NULL the receiver state of every receiver is
// computed into it in one pass (and kept), otherwise chunk by chunk in the workspace.
// With keep_mask non-zero, the state of the output groups in it is computed into `keep` (every
// receiver, group by group) and the other groups are streamed one group at a time.
int conv_fwd_impl(sobek_plan plan, sobek_graph graph, const float* x, const float* evec, const float* phi,
                  const float* W, float* out, float* state, void* ws, size_t ws_bytes, hipStream_t stream,
                  uint64_t keep_mask = 0, float* keep = nullptr, bool per_group = false) {
  int rc = check_common(plan, graph, x, evec, phi, W, ws, ws_bytes);
  if (rc) return rc;
  if (!out && graph->N) return fail(SOBEK_E_INVALID, "out is NULL");
  if (out && !aligned16(out)) return fail(SOBEK_E_ALIGN, "out is not 16-byte aligned");
  const Plan& p = plan->p;
  const sobek_graph_s& G = *graph;
  if (state && !aligned16(state)) return fail(SOBEK_E_ALIGN, "state is not 16-byte aligned");
  // the channelwise single-multiplicity forward keeps no receiver state unless asked to
  const bool state_free = p.mode == SOBEK_MODE_UVU && p.uvu_C > 0 && !state && !keep_mask;
  const bool groups_asked = per_group || keep_mask || p.policy == SOBEK_POLICY_PER_GROUP;
  WsPlan w;
  if ((rc = plan_workspace(p, G, SOBEK_PASS_FWD, ws_bytes, w, false,
                           state || keeps_all(p, keep_mask) ? 0 : (groups_asked && !state_free ? 1 : -1))))
    return rc;
  const bool by_group = !state && !state_free && (groups_asked || group_route_pays(p, w));
  if (G.N == 0) return SOBEK_OK;
  const bool mulir = p.layout == SOBEK_LAYOUT_MUL_IR;
  const float* xk = x;
  float* ok = out;
  if (mulir) {
    xk = (const float*)((char*)ws + w.off_x);
    ok = (float*)((char*)ws + w.off_out);
    if ((rc = transpose(p, x, (float*)xk, G.N, true, 0, stream))) return rc;
  }
  if (!state_free && (rc = ensure_receiver_route(plan))) return rc;
  if (by_group) {
    if ((rc = ensure_groups(plan)) ||
        (rc = fwd_by_group(p, G, w, ws, keep_mask, keep, true, xk, evec, phi, W, ok, stream)) ||
        (rc = zero_dead_out(p, ok, G.N, stream)))
      return rc;
    if (mulir && (rc = transpose(p, ok, out, G.N, false, 1, stream))) return rc;
    return SOBEK_OK;
  }
  if (state_free) {
    // channelwise, one multiplicity: every receiver at once, no receiver state
    int r0 = 0, n = (int)G.N;
    LAUNCH(p.k.uvu_fwd, cdiv(G.N, 4), cdiv(p.uvu_C, 64), 1, stream, (const int*)G.rowptr, (const int*)G.sender, evec,
           phi, xk, W, ok, r0, n, (const float*)nullptr);
    if ((rc = zero_dead_out(p, ok, G.N, stream))) return rc;
    if (mulir && (rc = transpose(p, ok, out, G.N, false, 1, stream))) return rc;
    return SOBEK_OK;
  }
  float* S = state ? state : state_ptr(w, ws, p, 0);  // a retained state is one chunk of all N receivers
  for (auto& c : w.chunks) {
    if ((rc = run_state(p, G, c, w, S, false, xk, evec, phi, nullptr, nullptr, nullptr, 0, stream))) return rc;
    if ((rc = run_mix(p, c, w, ws, S, W, ok, 0, stream))) return rc;
  }
  if ((rc = zero_dead_out(p, ok, G.N, stream))) return rc;
  if (mulir && (rc = transpose(p, ok, out, G.N, false, 1, stream))) return rc;
  return SOBEK_OK;
}

// Backward; with `state` non-NULL (the retained state of conv_fwd_impl) the weight
// gradient reads it in one pass instead of recomputing S chunk by chunk.
// With `adj_state` non-NULL the adjoint state Sbar = mbar A^T of every receiver is
// computed into it in one pass (and kept for a double backward); the edge kernel
// then reads each chunk's rows from it.
// With keep_mask non-zero the weight gradient reads the state of those output groups from `keep`
// (as sobek_conv_fwd_keep left it) and recomputes the others one group at a time.
int conv_bwd_impl(sobek_plan plan, sobek_graph graph, const float* x, const float* evec, const float* phi,
                  const float* W, const float* gout, const float* state, float* adj_state, float* gx, float* gevec,
                  float* gphi, float* gW, void* ws, size_t ws_bytes, hipStream_t stream, uint64_t keep_mask = 0,
                  const float* keep = nullptr) {
  int rc = check_common(plan, graph, x, evec, phi, W, ws, ws_bytes);
  if (rc) return rc;
  if (!gout && graph->N) return fail(SOBEK_E_INVALID, "gout is NULL");
  for (const void* q : {(const void*)gout, (const void*)gx, (const void*)gevec, (const void*)gphi, (const void*)gW})
    if (q && !aligned16(q)) return fail(SOBEK_E_ALIGN, "pointer %p is not 16-byte aligned", q);
  const Plan& p = plan->p;
  const sobek_graph_s& G = *graph;
  if (adj_state && !aligned16(adj_state)) return fail(SOBEK_E_ALIGN, "adj_state is not 16-byte aligned");
  WsPlan w;
  // the state slot holds S (weight gradient without a kept state) and Sbar (without a kept adjoint state)
  // (the state-free channelwise edge kernel reads mbar and A directly, no Sbar)
  const bool uvu_direct = p.mode == SOBEK_MODE_UVU && p.uvu_C > 0 && p.uvu_bwd_direct;
  // with it, A_bar comes from the edges directly (no receiver state; a kept S is not needed)
  const bool uvu_wg = uvu_direct && p.uvu_wgrad_direct;
  // the weight gradient one output group at a time: kept groups, or the per-group policy
  bool ga_groups = gW && !state && !uvu_wg && (keep_mask || p.policy == SOBEK_POLICY_PER_GROUP);
  const bool ga_recompute = gW && !state && !uvu_wg && !keeps_all(p, keep_mask);
  const bool need_slot = ga_recompute || (!uvu_direct && !adj_state && (gx || gevec || gphi));
  if ((!uvu_direct || (gW && !uvu_wg)) && (rc = ensure_receiver_route(plan))) return rc;
  if ((rc = plan_workspace(p, G, SOBEK_PASS_BWD, ws_bytes, w, false, need_slot ? 1 : 0))) return rc;
  if (gW && !state && !uvu_wg && group_route_pays(p, w)) ga_groups = true;
  if (gW) { if ((rc = fill_zero(p, gW, (int64_t)p.K * p.n_w, stream))) return rc; }
  if (G.N == 0) return SOBEK_OK;
  const bool mulir = p.layout == SOBEK_LAYOUT_MUL_IR;
  const float* xk = x;
  const float* gk = gout;
  float* gxk = gx;
  if (mulir) {
    xk = (const float*)((char*)ws + w.off_x);
    gk = (const float*)((char*)ws + w.off_gout);
    if (gx) gxk = (float*)((char*)ws + w.off_gx);
    if ((rc = transpose(p, x, (float*)xk, G.N, true, 0, stream))) return rc;
    if ((rc = transpose(p, gout, (float*)gk, G.N, false, 0, stream))) return rc;
  }
  float* S = state_ptr(w, ws, p, 0);
  float* Sb = S;  // the same slot: S is consumed by the weight-gradient GEMM first
  float* contrib = gx ? (float*)((char*)ws + w.off_contrib) : nullptr;
  const bool edge = gx || gevec || gphi;
  const Chunk all{0, (int)G.N, 0, G.E};
  // the weight gradient from a kept state shares nothing with the adjoint-state GEMM and the edge
  // windows that follow (its split partials have a region of their own): it runs beside them
  bool side_open = false;
  if (gW && state && !uvu_wg) {
    hipStream_t side = stream;
    if ((rc = side_fork(plan, stream, side))) return rc;
    side_open = true;
    if ((rc = run_ga(p, all, w, ws, state, G.N, gk, gW, true, true, side))) return rc;
  }
  if (gW && uvu_wg) {
    int na = 0, n = (int)G.N;
    for (size_t a = 0; a < p.in.size(); ++a)
      for (auto& q : p.paths)
        if (q.i_in == (int)a) { ++na; break; }
    float* P = (float*)((char*)ws + w.off_P);
    int rows = sobek::uvu_wgrad_waves(p.K, p.n_w);
    long long nw = (long long)p.K * p.n_w;
    LAUNCH(p.k.uvu_wgrad, rows / 4, p.uvu_NB, na, stream, (const int*)G.rowptr, (const int*)G.sender,
           evec, phi, xk, gk, P, n, (const float*)nullptr, rows);
    LAUNCH(p.k.uvu_wreduce, cdiv(nw, 256), 1, 1, stream, (const float*)P, rows, nw, gW);
  }
  if (ga_groups && ((rc = ensure_groups(plan)) ||
                    (rc = ga_by_group(p, G, w, ws, keep_mask, keep, xk, evec, phi, gk, gW, stream))))
    return rc;
  if (adj_state && (rc = run_sbar(p, all, G.N, gk, W, adj_state, stream))) return rc;
  bool first_win = true;  // the first edge window overall initialises the sender cursors and x-gradient rows
  for (size_t ci = 0; ci < w.chunks.size(); ++ci) {
    const Chunk& c = w.chunks[ci];
    if (gW && !state && !uvu_wg && !ga_groups) {
      if ((rc = run_state(p, G, c, w, S, false, xk, evec, phi, nullptr, nullptr, nullptr, 0, stream))) return rc;
      if ((rc = run_ga(p, c, w, ws, S, w.ncap, gk, gW, ci == 0, ci + 1 == w.chunks.size(), stream))) return rc;
    }
    if (edge) {
      if (!uvu_direct && !adj_state && (rc = run_sbar(p, c, w.ncap, gk, W, Sb, stream))) return rc;
      rc = for_edge_windows(G, c, w, [&](int64_t ea, int64_t eb, int ra, int nr) -> int {
        int e0 = (int)ea, e1 = (int)eb, flags = 0, sub_off = ra - c.r0;
        if (uvu_direct) {
          float* part = (float*)((char*)ws + w.off_contrib) + (size_t)w.ecap * p.dim_in;
          const int ns = p.uvu_sliced ? p.uvu_NA : 1;
          LAUNCH(p.k.uvu_bwd, cdiv(nr, 4), p.uvu_NB, ns, stream, (const int*)G.rowptr, (const int*)G.sender, evec,
                 phi, xk, W, gk, gphi, gevec, contrib, part, ra, nr, e0, e0, e1, (const float*)nullptr);
          if (p.uvu_NB * ns > 1 && (gphi || gevec))
            LAUNCH(p.k.uvu_bwd_fin, cdiv(eb - ea, 256), 1, 1, stream, evec, (const float*)part, gphi, gevec, e0, e1,
                   (const float*)nullptr);
        } else {
          long long ncap = w.ncap, sb_ncap = adj_state ? G.N : w.ncap;
          int sb_r0 = adj_state ? ra : sub_off;
          LAUNCH_N(p.k.bwd_E, 64 * p.adj_waves, nr, adj_edge_split(p, nr, eb - ea), 1, stream, (const int*)G.rowptr,
                   (const int*)G.sender, evec, phi, xk, (const float*)(adj_state ? adj_state : Sb),
                   (const float*)nullptr, (const float*)nullptr, (const float*)nullptr, (const float*)nullptr, gphi,
                   gevec, contrib, ra, nr, ncap, e0, flags, sb_ncap, sb_r0, e0, e1, sub_off);
        }
        const int first = first_win;
        first_win = false;
        return gx ? run_sender_reduce(p, G, ea, eb, w, ws, contrib, gxk, first, stream) : SOBEK_OK;
      });
      if (rc) return rc;
    }
  }
  if (gx && first_win && (rc = fill_zero(p, gxk, G.N * p.dim_in, stream))) return rc;  // no edges at all
  if (mulir && gx && (rc = transpose(p, gxk, gx, G.N, true, 1, stream))) return rc;
  if (side_open && (rc = side_join(plan, stream))) return rc;
  return SOBEK_OK;
}

}  // namespace

extern "C" {

int sobek_state_size(sobek_plan plan, sobek_graph graph, size_t* bytes) {
  if (!plan || !graph || !bytes) return fail(SOBEK_E_INVALID, "NULL argument");
  // fp32 elements for every plan: the same size serves the adjoint state (fp32), and a bf16 state
  // uses the first half
  *bytes = (size_t)graph->N * plan->p.srow * 4;
  return SOBEK_OK;
}

int sobek_conv_fwd(sobek_plan plan, sobek_graph graph, const float* x, const float* evec, const float* phi,
                   const float* W, float* out, void* ws, size_t ws_bytes, hipStream_t stream) {
  return conv_fwd_impl(plan, graph, x, evec, phi, W, out, nullptr, ws, ws_bytes, stream);
}

int sobek_conv_fwd_save(sobek_plan plan, sobek_graph graph, const float* x, const float* evec, const float* phi,
                        const float* W, float* out, float* state, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!state && graph && graph->N) return fail(SOBEK_E_INVALID, "state is NULL");
  return conv_fwd_impl(plan, graph, x, evec, phi, W, out, state, ws, ws_bytes, stream);
}

int sobek_conv_bwd(sobek_plan plan, sobek_graph graph, const float* x, const float* evec, const float* phi,
                   const float* W, const float* gout, float* gx, float* gevec, float* gphi, float* gW, void* ws,
                   size_t ws_bytes, hipStream_t stream) {
  return conv_bwd_impl(plan, graph, x, evec, phi, W, gout, nullptr, nullptr, gx, gevec, gphi, gW, ws, ws_bytes,
                       stream);
}

int sobek_plan_set_policy(sobek_plan plan, int policy) {
  if (!plan) return fail(SOBEK_E_INVALID, "NULL plan");
  if (policy != SOBEK_POLICY_ALL_GROUPS && policy != SOBEK_POLICY_PER_GROUP && policy != SOBEK_POLICY_AUTO)
    return fail(SOBEK_E_INVALID, "unknown scratch policy %d", policy);
  plan->p.policy = policy;
  return SOBEK_OK;
}

int sobek_kept_size(sobek_plan plan, sobek_graph graph, uint64_t group_mask, size_t* bytes) {
  if (!plan || !graph || !bytes) return fail(SOBEK_E_INVALID, "NULL argument");
  const Plan& p = plan->p;
  if (p.groups.size() < 64 && (group_mask >> p.groups.size()))
    return fail(SOBEK_E_INVALID, "group mask has bits past the plan's %zu output groups", p.groups.size());
  *bytes = kept_offset(p, graph->N, group_mask, (int)p.groups.size()) * state_elem(p);
  return SOBEK_OK;
}

int sobek_retention_select(sobek_plan plan, sobek_graph graph, size_t budget, uint64_t* group_mask, size_t* bytes) {
  if (!plan || !graph || !group_mask || !bytes) return fail(SOBEK_E_INVALID, "NULL argument");
  const Plan& p = plan->p;
  const size_t B = budget ? budget : default_budget();
  const int G = (int)std::min<size_t>(64, p.groups.size());
  std::vector<size_t> cost(G);
  std::vector<double> work(G, 0.0);
  for (int g = 0; g < G; ++g) {
    cost[g] = (size_t)graph->N * p.groups[g].d * p.groups[g].D * state_elem(p);
    for (int t : p.groups[g].paths) {
      size_t nz = 0;
      for (double c : p.paths[t].cg) nz += c != 0.0;
      work[g] += (double)nz * p.paths[t].c_in;
    }
  }
  uint64_t best = 0;
  const bool free_wgrad = p.mode == SOBEK_MODE_UVU && p.uvu_C > 0 && p.uvu_bwd_direct && p.uvu_wgrad_direct;
  if (free_wgrad) {
    best = 0;
  } else if (p.mode == SOBEK_MODE_UVU) {
    size_t all = 0;
    for (int g = 0; g < G; ++g) all += cost[g];
    if (G == (int)p.groups.size() && all <= B) best = G == 64 ? ~(uint64_t)0 : (((uint64_t)1 << G) - 1);
  } else if (G <= 20) {
    double bw = 0.0;
    size_t bb = 0;
    for (uint64_t m = 1; m < ((uint64_t)1 << G); ++m) {
      double v = 0.0;
      size_t b = 0;
      for (int g = 0; g < G; ++g)
        if (m >> g & 1) { v += work[g]; b += cost[g]; }
      if (b > B) continue;
      if (v > bw || (v == bw && b < bb)) { best = m; bw = v; bb = b; }
    }
  } else {
    std::vector<int> order(G);
    for (int g = 0; g < G; ++g) order[g] = g;
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) {
      return work[a] * (double)cost[b] > work[b] * (double)cost[a];
    });
    size_t used = 0;
    for (int g : order)
      if (used + cost[g] <= B) { best |= (uint64_t)1 << g; used += cost[g]; }
  }
  *group_mask = best;
  *bytes = kept_offset(p, graph->N, best, (int)p.groups.size()) * state_elem(p);
  return SOBEK_OK;
}

int sobek_conv_fwd_keep(sobek_plan plan, sobek_graph graph, const float* x, const float* evec, const float* phi,
                        const float* W, float* out, uint64_t group_mask, float* kept, void* ws, size_t ws_bytes,
                        hipStream_t stream) {
  if (!plan || !graph) return fail(SOBEK_E_INVALID, "NULL plan or graph");
  size_t kb = 0;
  if (int rc = sobek_kept_size(plan, graph, group_mask, &kb)) return rc;
  if (group_mask && graph->N && !kept) return fail(SOBEK_E_INVALID, "kept is NULL");
  if (kept && !aligned16(kept)) return fail(SOBEK_E_ALIGN, "kept is not 16-byte aligned");
  if (plan->p.mode == SOBEK_MODE_UVU && group_mask && !keeps_all(plan->p, group_mask))
    return fail(SOBEK_E_INVALID, "a channelwise plan keeps every output group or none");
  return conv_fwd_impl(plan, graph, x, evec, phi, W, out, nullptr, ws, ws_bytes, stream, group_mask, kept, true);
}

int sobek_conv_bwd_kept(sobek_plan plan, sobek_graph graph, const float* x, const float* evec, const float* phi,
                        const float* W, const float* gout, uint64_t group_mask, const float* kept, float* gx,
                        float* gevec, float* gphi, float* gW, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!plan || !graph) return fail(SOBEK_E_INVALID, "NULL plan or graph");
  size_t kb = 0;
  if (int rc = sobek_kept_size(plan, graph, group_mask, &kb)) return rc;
  if (group_mask && graph->N && gW && !kept) return fail(SOBEK_E_INVALID, "kept is NULL");
  if (kept && !aligned16(kept)) return fail(SOBEK_E_ALIGN, "kept is not 16-byte aligned");
  if (plan->p.mode == SOBEK_MODE_UVU && group_mask && !keeps_all(plan->p, group_mask))
    return fail(SOBEK_E_INVALID, "a channelwise plan keeps every output group or none");
  if (!gW) group_mask = 0;
  return conv_bwd_impl(plan, graph, x, evec, phi, W, gout, nullptr, nullptr, gx, gevec, gphi, gW, ws, ws_bytes,
                       stream, group_mask, group_mask ? kept : nullptr);
}

int sobek_materialized_workspace_size(sobek_plan plan, sobek_graph graph, size_t budget, size_t* bytes) {
  if (!plan || !graph || !bytes) return fail(SOBEK_E_INVALID, "NULL argument");
  const Plan& p = plan->p;
  if (!materialized_supported(p))
    return fail(SOBEK_E_UNSUPPORTED, "the materialized forward covers uvw plans in the ir_mul layout with fp32 GEMMs");
  const size_t per = materialized_edge_bytes(p);
  const size_t full = (size_t)std::max<int64_t>(1, graph->E) * per + 256;
  const size_t least = (size_t)std::max<int64_t>(1, graph->max_deg) * per + 256;
  *bytes = budget == 0 ? full : std::min(full, std::max(budget, least));
  return SOBEK_OK;
}

int sobek_conv_fwd_materialized(sobek_plan plan, sobek_graph graph, const float* x, const float* evec,
                                const float* phi, const float* W, float* out, void* ws, size_t ws_bytes,
                                hipStream_t stream) {
  int rc = check_common(plan, graph, x, evec, phi, W, ws, ws_bytes);
  if (rc) return rc;
  const Plan& p = plan->p;
  const sobek_graph_s& G = *graph;
  if (!materialized_supported(p))
    return fail(SOBEK_E_UNSUPPORTED, "the materialized forward covers uvw plans in the ir_mul layout with fp32 GEMMs");
  if (!out && G.N) return fail(SOBEK_E_INVALID, "out is NULL");
  if (out && !aligned16(out)) return fail(SOBEK_E_ALIGN, "out is not 16-byte aligned");
  if (G.N == 0) return SOBEK_OK;
  // the W block of the window's edges, then its M block (256-byte aligned)
  auto wbytes = [&](int64_t ne) { return ((size_t)ne * p.n_w * 4 + 255) / 256 * 256; };
  auto fits = [&](int64_t ne) { return wbytes(ne) + (size_t)ne * p.dim_out * 4 <= ws_bytes; };
  int64_t ecap = std::min<int64_t>((int64_t)(ws_bytes / materialized_edge_bytes(p)), kMatMaxWindow);
  while (ecap > 0 && !fits(ecap)) --ecap;
  if (G.E > 0 && ecap < std::max<int64_t>(1, G.max_deg))
    return fail(SOBEK_E_WORKSPACE, "workspace of %zu bytes holds %lld edges, fewer than the largest in-degree %lld",
                ws_bytes, (long long)ecap, (long long)G.max_deg);
  if ((rc = ensure_materialized(plan))) return rc;
  float* Wm = (float*)ws;
  float* Mm = (float*)((char*)ws + wbytes(std::max<int64_t>(0, ecap)));
  const int32_t* rp = G.h_rowptr.data();
  const unsigned colb = cdiv(p.dim_out, 256);
  const long long nw = p.n_w;
  for (int64_t r = 0; r < G.N;) {
    // whole receivers while their edges fit the window
    int64_t r1 = r + 1;
    while (r1 < G.N && rp[r1 + 1] - rp[r] <= ecap) ++r1;
    const long long e0 = rp[r];
    const int ne = (int)(rp[r1] - rp[r]);
    if (ne > 0) {
      LAUNCH(p.k.mat_w, cdiv(nw, 256), cdiv(ne, kMatEdgeTile), 1, stream, phi, W, Wm, e0, ne);
      LAUNCH(p.k.mat_msg, ne, 1, 1, stream, (const int*)G.sender, evec, x, (const float*)Wm, Mm, e0, ne);
    }
    const int r0 = (int)r, nr = (int)(r1 - r);
    LAUNCH(p.k.mat_reduce, nr, colb, 1, stream, (const int*)G.rowptr, (const float*)Mm, out, r0, nr, e0);
    r = r1;
  }
  return zero_dead_out(p, out, G.N, stream);
}

int sobek_conv_bwd_saved(sobek_plan plan, sobek_graph graph, const float* x, const float* evec, const float* phi,
                         const float* W, const float* gout, const float* state, float* adj_state, float* gx,
                         float* gevec, float* gphi, float* gW, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (state && !aligned16(state)) return fail(SOBEK_E_ALIGN, "state is not 16-byte aligned");
  return conv_bwd_impl(plan, graph, x, evec, phi, W, gout, state, adj_state, gx, gevec, gphi, gW, ws, ws_bytes,
                       stream);
}

}  // extern "C"

namespace {

// Double backward; with `adj_state` non-NULL (the adjoint state kept by
// sobek_conv_bwd_saved for the same gout and W) Sbar is read from it instead of
// being recomputed chunk by chunk.
int conv_dbwd_impl(sobek_plan plan, sobek_graph graph, const float* x, const float* evec, const float* phi,
                   const float* W, const float* gout, const float* adj_state, const float* t_gx, const float* t_gevec,
                   const float* t_gphi, const float* t_gW, float* g_gout, float* g_x, float* g_evec, float* g_phi,
                   float* g_W, void* ws, size_t ws_bytes, hipStream_t stream) {
  int rc = check_common(plan, graph, x, evec, phi, W, ws, ws_bytes);
  if (adj_state && !aligned16(adj_state)) return fail(SOBEK_E_ALIGN, "adj_state is not 16-byte aligned");
  if (rc) return rc;
  if (!gout && graph->N) return fail(SOBEK_E_INVALID, "gout is NULL");
  for (const void* q : {(const void*)gout, (const void*)t_gx, (const void*)t_gevec, (const void*)t_gphi,
                        (const void*)t_gW, (const void*)g_gout, (const void*)g_x, (const void*)g_evec,
                        (const void*)g_phi, (const void*)g_W})
    if (q && !aligned16(q)) return fail(SOBEK_E_ALIGN, "pointer %p is not 16-byte aligned", q);
  const Plan& p = plan->p;
  const sobek_graph_s& G = *graph;
  WsPlan w;
  const int flags = (t_gphi ? 1 : 0) | (t_gx ? 2 : 0) | (t_gevec ? 4 : 0) | (t_gW ? 8 : 0);
  // channelwise plans with the state-free kernels take the double backward of an edge-vector
  // cotangent alone without receiver state: m_dot, g_W and the edge terms along Ydot = J evd
  const bool uvu_free = p.mode == SOBEK_MODE_UVU && p.uvu_C > 0 && p.uvu_bwd_direct && p.uvu_wgrad_direct &&
                        p.uvu_tan_direct && flags == 4;
  if (!uvu_free && (rc = ensure_receiver_route(plan))) return rc;
  // the second state slot (Sbar') is needed only with a dA cotangent
  if ((rc = plan_workspace(p, G, SOBEK_PASS_DBWD, ws_bytes, w, false, uvu_free ? 0 : (t_gW ? 2 : 1)))) return rc;
  const bool tan = flags & 7;
  if (g_W) { if ((rc = fill_zero(p, g_W, (int64_t)p.K * p.n_w, stream))) return rc; }
  if (G.N == 0) return SOBEK_OK;
  const bool mulir = p.layout == SOBEK_LAYOUT_MUL_IR;
  const float *xk = x, *gk = gout, *txk = t_gx;
  float *ggk = g_gout, *gxk = g_x;
  if (mulir) {
    xk = (const float*)((char*)ws + w.off_x);
    gk = (const float*)((char*)ws + w.off_gout);
    if ((rc = transpose(p, x, (float*)xk, G.N, true, 0, stream))) return rc;
    if ((rc = transpose(p, gout, (float*)gk, G.N, false, 0, stream))) return rc;
    if (t_gx) {
      txk = (const float*)((char*)ws + w.off_tgx);
      if ((rc = transpose(p, t_gx, (float*)txk, G.N, true, 0, stream))) return rc;
    }
    if (g_gout) ggk = (float*)((char*)ws + w.off_out);
    if (g_x) gxk = (float*)((char*)ws + w.off_gx);
  }
  if (g_gout && !tan && !t_gW) { if ((rc = fill_zero(p, ggk, G.N * p.dim_out, stream))) return rc; }
  if (uvu_free) {
    int n = (int)G.N, r0 = 0;
    if (g_gout) {
      LAUNCH(p.k.uvu_fwd_t, cdiv(G.N, 4), p.uvu_NB, 1, stream, (const int*)G.rowptr, (const int*)G.sender, evec, phi,
             xk, W, ggk, r0, n, t_gevec);
      if ((rc = zero_dead_out(p, ggk, G.N, stream))) return rc;
    }
    if (g_W) {
      float* P = (float*)((char*)ws + w.off_P);
      int rows = sobek::uvu_wgrad_waves(p.K, p.n_w);
      long long nw = (long long)p.K * p.n_w;
      LAUNCH(p.k.uvu_wgrad_t, rows / 4, p.uvu_NB, p.uvu_NA, stream, (const int*)G.rowptr,
             (const int*)G.sender, evec, phi, xk, gk, P, n, t_gevec, rows);
      LAUNCH(p.k.uvu_wreduce, cdiv(nw, 256), 1, 1, stream, (const float*)P, rows, nw, g_W);
    }
    float* contrib = g_x ? (float*)((char*)ws + w.off_contrib) : nullptr;
    float* part = (float*)((char*)ws + w.off_contrib) + (size_t)w.ecap * p.dim_in;
    const int ns = p.uvu_sliced ? p.uvu_NA : 1;
    bool first_win = true;
    if (g_x || g_evec || g_phi)
      for (const Chunk& c : w.chunks) {
        rc = for_edge_windows(G, c, w, [&](int64_t ea, int64_t eb, int ra, int nr) -> int {
          int e0 = (int)ea, e1 = (int)eb;
          LAUNCH(p.k.uvu_bwd_t, cdiv(nr, 4), p.uvu_NB, ns, stream, (const int*)G.rowptr, (const int*)G.sender, evec,
                 phi, xk, W, gk, g_phi, g_evec, contrib, part, ra, nr, e0, e0, e1, t_gevec);
          if (p.uvu_NB * ns > 1 && (g_phi || g_evec))
            LAUNCH(p.k.uvu_bwd_fin_t, cdiv(eb - ea, 256), 1, 1, stream, evec, (const float*)part, g_phi, g_evec, e0,
                   e1, t_gevec);
          const int first = first_win;
          first_win = false;
          return g_x ? run_sender_reduce(p, G, ea, eb, w, ws, contrib, gxk, first, stream) : SOBEK_OK;
        });
        if (rc) return rc;
      }
    if (g_x && first_win && (rc = fill_zero(p, gxk, G.N * p.dim_in, stream))) return rc;
    if (mulir) {
      if (g_gout && (rc = transpose(p, ggk, g_gout, G.N, false, 1, stream))) return rc;
      if (g_x && (rc = transpose(p, gxk, g_x, G.N, true, 1, stream))) return rc;
    }
    return SOBEK_OK;
  }
  // one slot reused in stream order: dS (for m_dot and g_W), then S (for m_dot += S dA),
  // then Sbar; the second slot holds Sbar' when dA is active
  float* dS = state_ptr(w, ws, p, 0);
  float* S = dS;
  float* Sb = dS;
  float* Sb2 = state_ptr(w, ws, p, 1);
  float* contrib = g_x ? (float*)((char*)ws + w.off_contrib) : nullptr;
  const bool edge = g_x || g_evec || g_phi;
  // the state legs one output group at a time (per-group policy), then the edge legs by receiver chunk
  const bool by_group = p.policy == SOBEK_POLICY_PER_GROUP || group_route_pays(p, w);
  if (by_group && ((tan && (g_gout || g_W)) || (t_gW && g_gout)) &&
      ((rc = ensure_groups(plan)) ||
       (rc = dbwd_state_by_group(p, G, w, ws, xk, evec, phi, txk, t_gevec, t_gphi, flags, W, t_gW, gk,
                                 g_gout ? ggk : nullptr, g_W, stream))))
    return rc;
  bool first_win = true;  // the first edge window overall initialises the sender cursors and x-gradient rows
  // With the adjoint state kept and no dA cotangent, a chunk's dS GEMMs (m_dot = dS A, g_W += dS^T mbar)
  // share nothing with its edge windows (they read the kept adjoint state, not the slot): they run
  // beside them, and the next chunk's dS waits for them before it overwrites the slot.
  const bool overlap = adj_state && !t_gW && !by_group;
  bool side_open = false;
  for (size_t ci = 0; ci < w.chunks.size(); ++ci) {
    const Chunk& c = w.chunks[ci];
    if (tan && (g_gout || g_W) && !by_group) {
      if (side_open && (rc = side_join(plan, stream))) return rc;   // the slot's previous dS is consumed
      if ((rc = run_state(p, G, c, w, dS, true, xk, evec, phi, txk, t_gevec, t_gphi, flags & 7, stream))) return rc;
      hipStream_t gs = stream;
      if (overlap) {
        if ((rc = side_fork(plan, stream, gs))) return rc;
        side_open = true;
      }
      if (g_gout && (rc = run_mix(p, c, w, ws, dS, W, ggk, 0, gs))) return rc;
      if (g_W && (rc = run_ga(p, c, w, ws, dS, w.ncap, gk, g_W, ci == 0, ci + 1 == w.chunks.size(), gs)))
        return rc;
    }
    if (t_gW && g_gout && !by_group) {  // S reuses the slot once dS has been consumed
      if ((rc = run_state(p, G, c, w, S, false, xk, evec, phi, nullptr, nullptr, nullptr, 0, stream))) return rc;
      if ((rc = run_mix(p, c, w, ws, S, t_gW, ggk, tan ? 1 : 0, stream))) return rc;
    }
    if (edge) {
      if (!adj_state && (rc = run_sbar(p, c, w.ncap, gk, W, Sb, stream))) return rc;
      if (t_gW && (rc = run_sbar(p, c, w.ncap, gk, t_gW, Sb2, stream))) return rc;
      rc = for_edge_windows(G, c, w, [&](int64_t ea, int64_t eb, int ra, int nr) -> int {
        int e0 = (int)ea, e1 = (int)eb, fl = flags, sub_off = ra - c.r0;
        long long ncap = w.ncap, sb_ncap = adj_state ? G.N : w.ncap;
        int sb_r0 = adj_state ? ra : sub_off;
        LAUNCH_N(flags == 4 ? p.k.dbwd_E_r : p.k.dbwd_E, 64 * p.adj_waves, nr, adj_edge_split(p, nr, eb - ea), 1,
                 stream, (const int*)G.rowptr, (const int*)G.sender, evec, phi, xk,
                 (const float*)(adj_state ? adj_state : Sb), (const float*)Sb2, txk, t_gevec, t_gphi, g_phi, g_evec,
                 contrib, ra, nr, ncap, e0, fl, sb_ncap, sb_r0, e0, e1, sub_off);
        const int first = first_win;
        first_win = false;
        return g_x ? run_sender_reduce(p, G, ea, eb, w, ws, contrib, gxk, first, stream) : SOBEK_OK;
      });
      if (rc) return rc;
    }
  }
  if (g_x && first_win && (rc = fill_zero(p, gxk, G.N * p.dim_in, stream))) return rc;  // no edges at all
  if (side_open && (rc = side_join(plan, stream))) return rc;
  if (g_gout && (rc = zero_dead_out(p, ggk, G.N, stream))) return rc;
  if (mulir) {
    if (g_gout && (rc = transpose(p, ggk, g_gout, G.N, false, 1, stream))) return rc;
    if (g_x && (rc = transpose(p, gxk, g_x, G.N, true, 1, stream))) return rc;
  }
  return SOBEK_OK;
}

}  // namespace

extern "C" {

int sobek_conv_dbwd(sobek_plan plan, sobek_graph graph, const float* x, const float* evec, const float* phi,
                    const float* W, const float* gout, const float* t_gx, const float* t_gevec, const float* t_gphi,
                    const float* t_gW, float* g_gout, float* g_x, float* g_evec, float* g_phi, float* g_W, void* ws,
                    size_t ws_bytes, hipStream_t stream) {
  return conv_dbwd_impl(plan, graph, x, evec, phi, W, gout, nullptr, t_gx, t_gevec, t_gphi, t_gW, g_gout, g_x, g_evec,
                        g_phi, g_W, ws, ws_bytes, stream);
}

int sobek_conv_dbwd_saved(sobek_plan plan, sobek_graph graph, const float* x, const float* evec, const float* phi,
                          const float* W, const float* gout, const float* adj_state, const float* t_gx,
                          const float* t_gevec, const float* t_gphi, const float* t_gW, float* g_gout, float* g_x,
                          float* g_evec, float* g_phi, float* g_W, void* ws, size_t ws_bytes, hipStream_t stream) {
  return conv_dbwd_impl(plan, graph, x, evec, phi, W, gout, adj_state, t_gx, t_gevec, t_gphi, t_gW, g_gout, g_x,
                        g_evec, g_phi, g_W, ws, ws_bytes, stream);
}

}  // extern "C"
