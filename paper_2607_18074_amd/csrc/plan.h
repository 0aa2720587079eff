// Plan: the static description of one operator signature (irreps, K, layout,
// normalisation), the path/group/unit decomposition the kernels are generated
// from, and the compiled kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <array>
#include <cstdint>
#include <map>
#include <string>
#include <vector>

namespace sobek {

struct Irrep {
  int mul, l, p;
  int off;  // start in the flattened vector
  int dim() const { return mul * (2 * l + 1); }
};

// One tensor-product path (Section 2.4): input irrep a, SH order l_sh, output irrep c.
struct Path {
  int i_in, i_sh, i_out;
  int l_in, l_sh, l_out;
  int c_in, c_out;
  int64_t w_off = 0;    // offset in the flattened weight axis (eq. num_weights)
  double alpha = 1.0;   // path normalisation
  int group = -1;       // index into Plan::groups
  int64_t koff = 0;     // column offset of this path inside its group's receiver state
  std::vector<double> cg;  // alpha * Q, dense [d_in][d_sh][d_out]
};

// Output group g = one output irrep block with its paths (Section 4.2).
// Receiver state rows are (receiver, m_o); columns k = koff_pi + q * C_in + u.
struct Group {
  int i_out, l, d, C, off;
  std::vector<int> paths;
  int64_t D = 0;  // K * sum of C_in over the group's paths
  int64_t s_off = 0;  // per-receiver offset of the group block (floats) = sum of d*D of earlier groups
  int64_t ktab_off = 0;  // offset of this group's k-table in Plan::ktab
};

// A wave's share of the forward state kernel: input irrep a, channel block
// [U0, U0 + U) of the input multiplicity, ES edges in flight per wave
// (lane = sub * U + u), and the list of paths (all with input a).
struct Unit {
  int a;
  int U, U0, ES;
  std::vector<int> paths;
};

// Adjoint edge kernels: a wave takes 16 edges at a time.  Lane l holds edge
// slot l % 16 and the channel quad l / 16 of a 16-channel tile; the products
// with the staged adjoint state run on fp32 MFMA (16x16x4 for the q-contraction
// G = phi Sbar, 4x4x1 blocks for the channel contraction <Sbar, C>).  An item is
// (input irrep a, tile starting at channel u0, paths with input a); its
// adjoint-state slices are staged in LDS as [path][q < KP][m_o][16 channels].
struct AdjItem {
  int a, u0;
  std::vector<int> paths;
  bool first = true;          // first slab that writes (a, u0) contributions
  std::vector<int> lds_off;   // LDS offset (floats) of each path's slice
};

struct AdjSlab {
  std::vector<AdjItem> items;
  int floats = 0;
};

// The streaming adjoint-state GEMM stages the C-wide rows of 64 receivers-components in LDS
// (about 272*C + 17k bytes), so it serves output multiplicities up to 256; wider groups use
// the tiled sobek_gemm_sbar_64.
inline bool sbar_streams(bool vec4, int C) { return vec4 && C <= 256; }

// waves per slice of the state-free channelwise weight gradient, each writing one partial
// row of K * N_w floats: up to 1024 for occupancy, halved while the rows exceed 96 MiB (they
// share the per-edge contribution region of the workspace)
inline int uvu_wgrad_waves(int K, int64_t n_w) {
  int w = 1024;
  while (w > 64 && (int64_t)w * K * n_w * 4 > ((int64_t)96 << 20)) w >>= 1;
  return w;
}

struct Kernels {
  hipModule_t module = nullptr;    // every kernel of the plan (for channelwise plans with the
                                   // state-free kernels: the receiver-route kernels, loaded on first use)
  hipModule_t module_grp = nullptr;  // per-output-group state kernels (compiled on first use)
  std::vector<std::array<hipFunction_t, 3>> fwd_grp;  // per group: S, dS_r, dS
  hipModule_t module_mat = nullptr;  // the materialized-forward baseline (compiled on first use)
  hipFunction_t mat_w = nullptr, mat_msg = nullptr, mat_reduce = nullptr;
  hipModule_t module_u = nullptr;  // channelwise plans: the state-free kernels and the common ones
  hipFunction_t fwd_S = nullptr, fwd_dS = nullptr, fwd_dS_r = nullptr;
  hipFunction_t bwd_E = nullptr, dbwd_E = nullptr, dbwd_E_r = nullptr;
  hipFunction_t gemm_sa[3] = {}, gemm_sbar[3] = {}, gemm_ga[3] = {};  // BN = 16, 32, 64
  hipFunction_t gemm_sa_v[3] = {}, gemm_ga_v[3] = {}, gemm_sbar_v = nullptr;  // 16-byte aligned operands
  hipFunction_t gemm_sa_vb128 = nullptr;  // bf16-GEMM plans: m = S A for groups over 64 channels
  std::map<int, hipFunction_t> gemm_sbar_c;  // streaming adjoint-state GEMM per output multiplicity
  hipFunction_t ga_reduce = nullptr, sender_reduce = nullptr, transpose = nullptr, fill_cols = nullptr,
                zero = nullptr, sa_reduce = nullptr;
  hipFunction_t uvu_mix = nullptr, uvu_sbar = nullptr, uvu_ga = nullptr;  // channelwise mixing
  hipFunction_t uvu_fwd = nullptr, uvu_bwd = nullptr, uvu_bwd_fin = nullptr;  // channelwise state-free kernels
  hipFunction_t uvu_wgrad = nullptr, uvu_wreduce = nullptr;
  hipFunction_t uvu_fwd_t = nullptr, uvu_bwd_t = nullptr, uvu_bwd_fin_t = nullptr, uvu_wgrad_t = nullptr;  // tangent
};

struct Plan {
  std::vector<Irrep> in, out;
  int lmax = 0, K = 0, layout = 0, dtype = 0, norm = 0;
  int mode = 0;                 // 0: uvw (fully connected mixing), 1: uvu (channelwise)
  int policy = 2;               // scratch policy: 0 all groups per receiver chunk, 1 one output group at a
                                // time, 2 (default) the second when the first gives three or more chunks
                                // too small to fill the GPU
  std::vector<int> grp_units;   // forward wave units of each output group's own state kernels
  int dim_in = 0, dim_out = 0, nsh = 0;
  int64_t n_w = 0;
  std::vector<Path> paths;
  std::vector<Group> groups;
  int64_t srow = 0;  // floats of receiver state per receiver (sum over groups of d * D)
  std::vector<int32_t> ktab;   // host copy of all groups' k-tables
  std::vector<Unit> fwd_units;
  int adj_U = 16;               // channels per adjoint tile
  int adj_KP = 4;               // K rounded up to a multiple of 4
  int adj_waves = 2;            // waves per adjoint block (16 edges each per iteration)
  std::vector<AdjSlab> slabs;
  int bwd_eb = 64;              // edges per batch when the adjoint state needs several slabs
  int bwd_lds_max = 0;          // largest slab (floats)
  bool vec4 = false;            // every multiplicity a multiple of 4: vectorised GEMMs apply
  int uvu_C = 0;                // uvu with one multiplicity C on every path: the state-free kernels apply
  int uvu_NB = 0;               // 64-channel blocks of C
  int uvu_NA = 0;               // input irreps with paths (slices of the state-free backward)
  bool uvu_bwd_direct = false;  // the state-free backward compiled without register spills (set at load)
  bool uvu_sliced = false;      // ... in its per-input-irrep form (the all-irrep form spilled)
  bool uvu_wgrad_direct = false;  // likewise the state-free weight gradient
  bool uvu_tan_direct = false;    // and their edge-vector-tangent variants (double backward)
  std::vector<int> dead_in;     // input irreps no path reads (their gradients are zero)
  std::vector<int> dead_out;    // output irreps no path writes (their outputs are zero)
  std::string source;           // generated HIP source
  std::string source_u;         // channelwise plans with the state-free kernels: that part alone
  bool rr_loaded = false;       // the receiver-route kernels are loaded
  std::string cache_key;
  Kernels k;
  // device tables
  int32_t* d_ktab = nullptr;
  int32_t* d_in_blocks = nullptr;   // [3][n_in]: off, mul, dim(2l+1)
  int32_t* d_out_blocks = nullptr;  // [3][n_out]
};

// Builds paths, groups, units and slabs for a validated signature.
void build_plan(Plan& p);
// Generates the plan-specific HIP source (prepended by the shared prelude at compile time).
std::string generate_source(const Plan& p, bool receiver_route = true);
// bf16-GEMM plans run the streaming adjoint-state GEMM on bf16 MFMA for output multiplicities in
// multiples of 32 up to 128 (sobek_gemm_sbar_cb<C>, 256 rows of mbar per block); other widths keep
// the fp32 kernels (64 rows per block).
inline bool sbar_bf16(const Plan& p, int C) { return p.dtype == 1 && sbar_streams(p.vec4, C) && C % 32 == 0 && C <= 128; }
inline int sbar_block_rows(const Plan& p, int C) { return sbar_bf16(p, C) ? 256 : 64; }

// Source of the materialized-forward baseline module (Section 2.4, eq. radial_projection_background).
std::string generate_materialized_source(const Plan& p);
// Source of the per-output-group state kernels (Appendix B.2, eq. receiver_chunk_budget).
std::string generate_group_source(const Plan& p);
// Forward wave units over every path (group < 0) or over the paths into one output group.
std::vector<Unit> pack_fwd_units(const Plan& p, int group, std::vector<int>* dead_in);

}  // namespace sobek
