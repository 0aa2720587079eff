/*
 * sobek.h -- C ABI of libsobek_hip: the edge-conditioned Clebsch-Gordan
 * tensor-product convolution with fully connected (uvw) multiplicity mixing,
 * forward, backward and double backward, on AMD Instinct MI355X (gfx950).
 *
 * Operator (arXiv 2607.18074, Section 2.4, eqs. standard_tpconv_background
 * and radial_projection_background): for every receiver i of a directed graph,
 *
 *   m_i = sum_{e = (j -> i)} sum_{paths pi} sum_{u, w}
 *           ( sum_q phi[e, q] W[q, off_pi + u C_out + w] )
 *           * sum_{m_i, m_y} c^pi[m_i, m_y, m_o] x_j[u, m_i] Y_e[m_y]
 *
 * where Y_e are real spherical harmonics of the edge vector evec[e]
 * (component normalised, m = -l..l, Y_1 = sqrt3 (y, z, x)) and c^pi is the
 * real-basis Clebsch-Gordan tensor of the path (Section 4.2, eq.
 * angular_path_contraction) times the path normalisation.  The library
 * evaluates it in the receiver-factorised streaming order of Sections 4.2-4.4
 * (eqs. receiver_state, receiver_matrix_product, receiver_adjoint,
 * receiver_double_adjoint): per-edge weights W_e = phi_e A, per-edge messages
 * and per-edge weight adjoints are never written to device memory.
 *
 * Conventions shared by every call
 * --------------------------------
 * Status: every function returns 0 (SOBEK_OK) or a negative sobek_status.
 *   sobek_last_error() returns a message for the last failure on the calling
 *   thread; the pointer stays valid until the next sobek_* call on that thread.
 * Memory: every device pointer is caller-owned.  conv_* calls never allocate
 *   device memory; their scratch is the caller's workspace (ws, ws_bytes).
 *   Plans own small device tables allocated in sobek_plan_create.  The one
 *   exception is code: a channelwise plan with the state-free kernels loads
 *   only those at creation, and the first conv_* call that needs its
 *   receiver-route kernels (a forward that keeps its state, a weight gradient
 *   or double backward that cannot take the state-free route) compiles them
 *   (hipRTC, or the on-disk cache) and loads them, which allocates device
 *   memory for the code and may take seconds.
 * Streams: conv_* calls enqueue work on the given stream and return without
 *   synchronising.  They overwrite their outputs (no accumulation).
 * Determinism: for identical inputs, plan, graph and workspace size the
 *   results are bitwise identical (fixed reduction orders, no float atomics).
 * Validation: shapes, null pointers, alignment and workspace size are checked
 *   on the host.  Graph contents are validated by sobek_graph_prepare.
 *   Zero-length edge vectors are a precondition violation (undefined result).
 * Layouts (row-major, fp32):
 *   x, gx      [N][dim_in]   irrep blocks in descriptor order; within a block
 *              of multiplicity C and order l, element (u, m) sits at
 *              off + m*C + u  (SOBEK_LAYOUT_IR_MUL) or off + u*(2l+1) + m
 *              (SOBEK_LAYOUT_MUL_IR).
 *   out, gout  [N][dim_out]  same convention with the output irreps.
 *   evec       [E][3]        r_sender - r_receiver, receiver-sorted edge order.
 *   phi        [E][K]        radial / invariant edge features, same order.
 *   W          [K][n_weights] path-major in path order, then u, then w.
 */
#ifndef SOBEK_H_
#define SOBEK_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum sobek_status {
  SOBEK_OK = 0,
  SOBEK_E_INVALID = -1,     /* bad argument value or descriptor */
  SOBEK_E_UNSUPPORTED = -2, /* valid request the library does not implement (e.g. l > 3) */
  SOBEK_E_SHAPE = -3,       /* sizes inconsistent with the plan or graph */
  SOBEK_E_ALIGN = -4,       /* a pointer is not 16-byte aligned */
  SOBEK_E_WORKSPACE = -5,   /* workspace missing or smaller than the minimum */
  SOBEK_E_HIP = -6,         /* a HIP runtime call failed (message has the HIP error) */
  SOBEK_E_INTERNAL = -7,    /* internal invariant violated */
  SOBEK_E_COMPILE = -8      /* kernel generation or hipRTC compilation failed */
} sobek_status;

enum { SOBEK_LAYOUT_IR_MUL = 0, SOBEK_LAYOUT_MUL_IR = 1 };
enum { SOBEK_DTYPE_F32 = 0, SOBEK_DTYPE_BF16_GEMM = 1 };
enum { SOBEK_NORM_NONE = 0, SOBEK_NORM_FAN_IN = 1 };
enum { SOBEK_MODE_UVW = 0, SOBEK_MODE_UVU = 1 };
enum { SOBEK_POLICY_ALL_GROUPS = 0, SOBEK_POLICY_PER_GROUP = 1, SOBEK_POLICY_AUTO = 2 };
enum { SOBEK_PASS_FWD = 0, SOBEK_PASS_BWD = 1, SOBEK_PASS_DBWD = 2 };

/* One irreducible representation: multiplicity, order l >= 0, parity +1 ('e') or -1 ('o'). */
typedef struct sobek_irrep {
  int32_t mul, l, parity;
} sobek_irrep;

typedef struct sobek_plan_s *sobek_plan;   /* opaque; owns device tables and compiled kernels */
typedef struct sobek_graph_s *sobek_graph; /* opaque; host metadata + views into a caller buffer */

const char *sobek_last_error(void);
int sobek_version(void);

/* Plan: paths, tables and kernels for one operator signature.
 *   in[n_in], out[n_out]: input and output irreps (mul >= 1, 0 <= l <= 3).
 *   lmax: spherical harmonics 1x0e + 1x1o + ... up to lmax (<= 3), parity (-1)^l.
 *   K: radial width (1..64).
 *   mode: SOBEK_MODE_UVW, fully connected channel mixing (eq. uvw_connection):
 *         a path owns C_in*C_out weights, W[q][w_off + u*C_out + w];
 *         SOBEK_MODE_UVU, channelwise (eq. uvu_connection): every path needs
 *         C_out = C_in (else SOBEK_E_INVALID) and owns C_in weights,
 *         W[q][w_off + u], output channel u = input channel u.
 *   layout: SOBEK_LAYOUT_*.
 *   dtype: SOBEK_DTYPE_F32, fp32 throughout (the paper's precision, Section 5.1);
 *          SOBEK_DTYPE_BF16_GEMM, a reduced-precision option for uvw plans whose
 *          multiplicities are all multiples of 4 (else SOBEK_E_UNSUPPORTED): the
 *          channel GEMMs, m = S A (Section 4.2 eq. receiver_matrix_product; the
 *          forward, and the double backward's products with S and dS), A_bar =
 *          S^T mbar (Section 4.3 eq. receiver_adjoint; the weight gradients) and,
 *          for output groups whose multiplicity is a multiple of 32 (up to 128),
 *          the adjoint state Sbar = mbar A^T (same equation; the backward's and
 *          double backward's edge terms read it), round both operands to bf16
 *          (nearest even) and accumulate in fp32 on bf16 MFMA.  Every tensor at
 *          this boundary stays fp32; S is stored in bf16, Sbar in fp32; the edge
 *          stage and every reduction stay fp32.
 *   (uvu plans whose paths share one multiplicity run a forward and backward
 *   without receiver state; the environment variable SOBEK_UVU_ROUTE=receiver,
 *   read at plan creation, keeps them on the receiver-state route instead.
 *   Their backward edge kernel has two forms, all input irreps per lane or one
 *   input irrep per slice, chosen at plan creation from the compiled kernels'
 *   register and scratch use; SOBEK_UVU_FORM=u or SOBEK_UVU_FORM=s, read at
 *   plan creation, forces the first or the second, for testing.)
 *   path_norm: SOBEK_NORM_NONE (alpha = 1) or SOBEK_NORM_FAN_IN
 *   (alpha = 1/sqrt(fan_in), fan_in = number of terms summed into one output
 *   channel: the sum of C_in over the paths into the same output irrep for
 *   uvw, the number of such paths for uvu).
 * Paths are every (input, SH, output) triple allowed by the selection rules
 * of Section 2.2 (eq. cg_selection_rules), in lexicographic index order, with
 * weight offsets w_off in that order (eq. num_weights).  Kernels are generated
 * for the signature and compiled with hipRTC for gfx950 (cached on disk).  The
 * plan must be destroyed with sobek_plan_destroy. */
int sobek_plan_create(const sobek_irrep *in, int n_in, int lmax, const sobek_irrep *out, int n_out,
                      int K, int mode, int layout, int dtype, int path_norm, sobek_plan *plan);
int sobek_plan_destroy(sobek_plan plan);
/* Generate and compile (hipRTC, gfx950) the kernels of a signature into the
 * on-disk code-object cache without touching a GPU; arguments as in
 * sobek_plan_create.  Lets a build step prepare kernels ahead of a GPU run.
 * Channelwise plans with the state-free kernels load those at creation and the
 * receiver-route kernels on first use (a double backward with cotangents other
 * than the edge vectors', a forward that keeps its state); both are compiled
 * here, or only the first with SOBEK_JIT_STATE_FREE_ONLY=1 in the environment.
 * SOBEK_JIT_GROUPS=1 also compiles the per-output-group state kernels
 * (sobek_plan_set_policy, sobek_conv_fwd_keep). */
int sobek_jit_compile(const sobek_irrep *in, int n_in, int lmax, const sobek_irrep *out, int n_out, int K,
                      int mode, int layout, int dtype, int path_norm);
/* Full HIP source generated for a signature (prelude + plan code), NUL-terminated
 * into buf when buf_bytes allows; *needed gets the size including the NUL. */
int sobek_plan_source(const sobek_irrep *in, int n_in, int lmax, const sobek_irrep *out, int n_out, int K,
                      int mode, int layout, int dtype, int path_norm, char *buf, size_t buf_bytes, size_t *needed);
/* Sizes of the plan; any output pointer may be NULL. */
int sobek_plan_info(sobek_plan plan, int64_t *n_paths, int64_t *n_weights, int64_t *dim_in,
                    int64_t *dim_out, int64_t *dim_sh);
/* Path table (host arrays of n_paths entries; any may be NULL). */
int sobek_plan_paths(sobek_plan plan, int32_t *i_in, int32_t *i_sh, int32_t *i_out, int64_t *w_offset);
/* Dense copy of c^pi for path `path` into the host array
 * coeff[(2l_in+1)*(2l_sh+1)*(2l_out+1)], index (m_i, m_y, m_o) row-major. */
int sobek_plan_cg(sobek_plan plan, int path, double *coeff);
/* Generator's real coupling tensor Q for (l1, l2, l3) (no path normalisation) into the host array
 * coeff[(2l1+1)*(2l2+1)*(2l3+1)], index (a, b, c) row-major.  Needs no GPU. */
int sobek_cg_table(int l1, int l2, int l3, double *coeff);
/* Spherical-harmonic table of the generator: Y_lm(u) = sum_t coeff[t] ux^p[t][0] uy^p[t][1] uz^p[t][2]
 * on the unit sphere.  Writes at most max_terms terms; *n_terms gets the count. */
int sobek_sh_table(int l, int m, int32_t *n_terms, double *coeff, int32_t *powers, int max_terms);

/* Graph preparation (outside any timed region).  Inputs are the
 * receiver-sorted CSR on the device: recv_rowptr[N+1] (int32, non-decreasing,
 * recv_rowptr[0] = 0, recv_rowptr[N] = E) and sender[E] (int32 in [0, N)).
 * The call validates them, builds the stable sender-sorted view (Section 4.3:
 * one fixed reduction order per source row) into the caller's device buffer
 * buf (at least sobek_graph_prepare_size bytes, 16-byte aligned) and keeps a
 * host copy of recv_rowptr.  It synchronises the stream.  The CSR arrays and
 * buf must outlive the graph handle. */
int sobek_graph_prepare_size(int64_t N, int64_t E, size_t *bytes);
int sobek_graph_prepare(const int32_t *recv_rowptr, const int32_t *sender, int64_t N, int64_t E,
                        void *buf, size_t bytes, sobek_graph *graph, hipStream_t stream);
int sobek_graph_destroy(sobek_graph graph);
/* Number of nodes and edges of a prepared graph (either pointer may be NULL). */
int sobek_graph_info(sobek_graph graph, int64_t *N, int64_t *E);

/* Workspace for one pass (Section 4.2: receiver state and chunk buffers stay
 * within a fixed scratch budget and never scale with the edge count; the
 * Appendix on the runtime scratch budget).  The bytes of a single chunk over every receiver when
 * that fits in `budget` (budget 0 = the default of 1 GiB), else `budget` itself
 * (or the minimum for chunks of one receiver, if larger), so that a call given
 * exactly the reported bytes chunks as finely as the budget requires and no
 * finer.  The bytes never scale with E * n_weights or E * dim_out: receiver
 * state is bounded by the chunk size, per-edge x-gradient contributions by the
 * chunk's edges.  conv_* derive their chunking from ws_bytes.  For the double
 * backward of a channelwise plan with the state-free kernels the figure covers
 * both routes a call may take (receiver state for general cotangents, none for
 * an edge-vector cotangent alone). */
int sobek_workspace_size(sobek_plan plan, sobek_graph graph, int pass, size_t budget, size_t *bytes);

/* Streams: every conv_* call queues its work on `stream` and returns without synchronising.  Some
 * calls run part of it on a second stream of the plan (the backward's weight gradient from a kept
 * state, the double backward's dS GEMMs when the adjoint state is kept), forked from `stream` and
 * joined back into it with events, so everything the call writes is ready for later work on
 * `stream`; calls on one plan from several threads serialise that part. */

/* Forward (Section 4.2): out[N][dim_out] = conv(x, evec, phi, W). */
int sobek_conv_fwd(sobek_plan plan, sobek_graph graph, const float *x, const float *evec,
                   const float *phi, const float *W, float *out, void *ws, size_t ws_bytes,
                   hipStream_t stream);

/* Backward (Sections 3.2 and 4.3): gradients of <gout, conv(...)> with respect
 * to x [N][dim_in], evec [E][3], phi [E][K] and W [K][n_weights].  Any output
 * may be NULL when not needed. */
int sobek_conv_bwd(sobek_plan plan, sobek_graph graph, const float *x, const float *evec,
                   const float *phi, const float *W, const float *gout, float *gx, float *gevec,
                   float *gphi, float *gW, void *ws, size_t ws_bytes, hipStream_t stream);

/* Retained receiver state (Section 4.3: the weight gradient needs S; it is kept
 * from the forward when it fits, else recomputed).  sobek_state_size gives the
 * bytes of the state of every receiver of a graph: N * (sum over output groups
 * of (2l+1) * K * sum of C_in of the group's paths) floats, in a library-defined
 * order that callers treat as opaque.  It is bounded by the node count, never
 * by the edge count.  Plans with SOBEK_DTYPE_BF16_GEMM store S (not Sbar) in
 * bf16 and use the first half of such a buffer.
 *
 * sobek_conv_fwd_save is sobek_conv_fwd that also leaves S of every receiver in
 * `state` (caller-owned device memory of sobek_state_size bytes, 16-byte
 * aligned; overwritten).
 *
 * sobek_conv_bwd_saved is sobek_conv_bwd with two optional state buffers of
 * sobek_state_size bytes each (NULL = not used):
 *   state      read: the weight gradient takes S from it instead of
 *              recomputing it; it must come from sobek_conv_fwd_save with the
 *              same plan, graph, x, evec and phi (W may differ: S does not
 *              depend on it);
 *   adj_state  written: the adjoint state Sbar = gout A^T (Section 4.3, eq.
 *              receiver_adjoint) of every receiver, computed once and kept,
 *              so that a double backward with the same gout and W need not
 *              recompute it.
 * sobek_conv_dbwd_saved is sobek_conv_dbwd that reads Sbar from such an
 * adj_state (same plan, graph, gout and W) instead of recomputing it.
 * All take the workspace of their pass (sobek_workspace_size with the pass
 * constant); results agree with the plain calls within rounding (the weight
 * gradient's summation splits differ). */
int sobek_state_size(sobek_plan plan, sobek_graph graph, size_t *bytes);

/* Scratch policy of a plan's receiver-state legs (Appendix B.2, eq. receiver_chunk_budget).
 * SOBEK_POLICY_ALL_GROUPS: each receiver chunk builds the state of every output group, in chunks
 * sized by the workspace planner.  SOBEK_POLICY_AUTO (the default): per pass, the per-group route
 * below when the all-group plan of the pass needs three or more receiver chunks (Appendix B.2 takes
 * a chunked route only when it gives at least three chunks) and each chunk holds fewer than 8192
 * forward-state waves (receivers x wave units: too few to fill the GPU), else all groups; the
 * per-group route walks every edge once per output group.
 * SOBEK_POLICY_PER_GROUP: the forward, the
 * backward's weight gradient and the double backward's state legs (dS and S) take one output
 * group g at a time, in chunks of n_g = min(N, max(1, floor(B / (4 d_g (D_g + C_g))))) receivers,
 * with B the bytes of the pass workspace's receiver-state region (d_g = 2l+1, D_g the group's
 * state width, C_g its output multiplicity); the adjoint edge legs keep all-group receiver chunks.
 * Workspace sizes do not change.  Results agree with the default within rounding (the channel
 * GEMMs' split sums follow the chunk sizes) and are deterministic for a given policy and workspace
 * size.  The per-group kernels are compiled (hipRTC or the on-disk cache) and loaded on first use.
 * Not thread-safe against calls running on the plan. */
int sobek_plan_set_policy(sobek_plan plan, int policy);

/* Retention of complete output groups (Section 4.2: forward state is kept only as whole output
 * groups within the scratch budget, the others recomputed over bounded receiver ranges; Appendix
 * B.2).  A kept state for `group_mask` (bit g = output group g: the g-th output irrep, in order,
 * that some path reaches; groups past the 64th cannot be kept) holds, group by group in that order, the N d_g D_g state elements of
 * each kept group: fp32, or bf16 for SOBEK_DTYPE_BF16_GEMM plans.
 * sobek_kept_size: its bytes (SOBEK_E_INVALID for mask bits past the plan's groups).
 * sobek_retention_select: the paper's choice within `budget` bytes (0 = 1 GiB): for uvw plans the
 * subset of groups whose kept bytes fit and that avoids the most recomputed coupling work (the
 * sum over the group's paths of the non-zero coefficients times C_in), ties to fewer bytes (exact
 * over all subsets up to 20 groups, else groups taken greedily by work per byte); for uvu plans
 * every group when all fit, else none; none for channelwise plans whose weight gradient is
 * state-free.  *bytes gets the kept bytes of the chosen mask.
 * sobek_conv_fwd_keep: sobek_conv_fwd that writes the state of the groups of `group_mask` into
 * `kept` (caller-owned device memory of sobek_kept_size bytes, 16-byte aligned; overwritten) and
 * streams the other groups one group at a time as SOBEK_POLICY_PER_GROUP does.
 * sobek_conv_bwd_kept: sobek_conv_bwd whose weight gradient reads those groups from `kept` (written
 * by sobek_conv_fwd_keep with the same plan, graph, mask, x, evec and phi) and recomputes the others
 * one group at a time; gW NULL leaves `kept` unread.
 * Both take the workspace of their pass (sobek_workspace_size); results agree with the plain calls
 * within rounding.  Channelwise (uvu) plans keep every group or none (else SOBEK_E_INVALID). */
int sobek_kept_size(sobek_plan plan, sobek_graph graph, uint64_t group_mask, size_t *bytes);
int sobek_retention_select(sobek_plan plan, sobek_graph graph, size_t budget, uint64_t *group_mask,
                           size_t *bytes);
int sobek_conv_fwd_keep(sobek_plan plan, sobek_graph graph, const float *x, const float *evec,
                        const float *phi, const float *W, float *out, uint64_t group_mask, float *kept,
                        void *ws, size_t ws_bytes, hipStream_t stream);
int sobek_conv_bwd_kept(sobek_plan plan, sobek_graph graph, const float *x, const float *evec,
                        const float *phi, const float *W, const float *gout, uint64_t group_mask,
                        const float *kept, float *gx, float *gevec, float *gphi, float *gW, void *ws,
                        size_t ws_bytes, hipStream_t stream);

/* Materialized forward (Section 2.4 eq. radial_projection_background and the edge
 * messages of Section 2.5): the conventional evaluation order, kept as a comparison
 * system for the memory law of Section 2.5 (eq. uvw_width_scaling) and as a second route
 * to the forward.  It forms the per-edge weights W = phi A (E x N_w floats) and the per-edge
 * messages M (E x dim_out floats) in the workspace, then sums M over each receiver's edges;
 * the result equals sobek_conv_fwd's up to rounding.  Fully connected (uvw) plans in the
 * ir_mul layout with fp32 GEMMs only (else SOBEK_E_UNSUPPORTED).
 * sobek_materialized_workspace_size: budget 0 gives the bytes of W and M for every edge
 * (E x (N_w + dim_out) x 4, the materialized memory); a budget gives that much (or one
 * receiver's edges at the largest in-degree, if more), and the call then processes whole
 * receivers in edge windows that fit.  sobek_conv_fwd_materialized takes the same inputs as
 * sobek_conv_fwd (device pointers, 16-byte aligned) and fails with SOBEK_E_WORKSPACE when the
 * workspace cannot hold the edges of the receiver with the largest in-degree.  The kernels
 * are compiled (hipRTC or the on-disk cache) and loaded on the plan's first call. */
int sobek_materialized_workspace_size(sobek_plan plan, sobek_graph graph, size_t budget, size_t *bytes);
int sobek_conv_fwd_materialized(sobek_plan plan, sobek_graph graph, const float *x, const float *evec,
                                const float *phi, const float *W, float *out, void *ws, size_t ws_bytes,
                                hipStream_t stream);
int sobek_conv_fwd_save(sobek_plan plan, sobek_graph graph, const float *x, const float *evec,
                        const float *phi, const float *W, float *out, float *state, void *ws,
                        size_t ws_bytes, hipStream_t stream);
int sobek_conv_bwd_saved(sobek_plan plan, sobek_graph graph, const float *x, const float *evec,
                         const float *phi, const float *W, const float *gout, const float *state,
                         float *adj_state, float *gx, float *gevec, float *gphi, float *gW, void *ws,
                         size_t ws_bytes, hipStream_t stream);
int sobek_conv_dbwd_saved(sobek_plan plan, sobek_graph graph, const float *x, const float *evec,
                          const float *phi, const float *W, const float *gout, const float *adj_state,
                          const float *t_gx, const float *t_gevec, const float *t_gphi, const float *t_gW,
                          float *g_gout, float *g_x, float *g_evec, float *g_phi, float *g_W, void *ws,
                          size_t ws_bytes, hipStream_t stream);

/* Double backward (Sections 3.3 and 4.4): vector-Jacobian product of the
 * backward map (gout, x, evec, phi, W) -> (gx, gevec, gphi, gW) with
 * cotangents t_gx [N][dim_in], t_gevec [E][3], t_gphi [E][K], t_gW [K][n_weights]
 * (NULL = zero).  Outputs: g_gout [N][dim_out] (the tangent output),
 * g_x, g_evec, g_phi, g_W; any may be NULL.  g_evec includes the
 * spherical-harmonic Hessian term sum_m Ybar_m Hess(Y_m) t_gevec. */
int sobek_conv_dbwd(sobek_plan plan, sobek_graph graph, const float *x, const float *evec,
                    const float *phi, const float *W, const float *gout, const float *t_gx,
                    const float *t_gevec, const float *t_gphi, const float *t_gW, float *g_gout,
                    float *g_x, float *g_evec, float *g_phi, float *g_W, void *ws, size_t ws_bytes,
                    hipStream_t stream);

/* Measurement instrumentation (not part of the operator).  When enabled, each
 * kernel launch of the library is bracketed by two hipEvents recorded on the
 * launch stream.  sobek_profile_query synchronises on those events and reports,
 * per kernel name (index idx in name order), the launch count and summed
 * event-to-event milliseconds; it returns SOBEK_E_INVALID past the last name.
 * sobek_profile_reset drops the records.  Not thread-safe against concurrent
 * launches on other threads while enabled. */
int sobek_profile_enable(int on);
int sobek_profile_reset(void);
int sobek_profile_query(int idx, char *name, size_t name_bytes, int64_t *launches, double *total_ms);

#ifdef __cplusplus
}
#endif

#endif /* SOBEK_H_ */
