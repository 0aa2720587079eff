// Device code shared by every generated plan.  The plan generator prepends its
// constants and specialised edge kernels to this file and compiles the result
// with hipRTC for gfx950 (wave64, fp32 MFMA, packed-FP32 disabled).
//
// Contents
//   * channel GEMMs on fp32 MFMA (v_mfma_f32_16x16x4_f32), per output group g
//     of the receiver-factorised program (Section 4.2 eq. receiver_matrix_product,
//     Section 4.3 eq. receiver_adjoint, Section 4.4 eq. receiver_double_adjoint):
//       sobek_gemm_sa    out(i, m_o, w)  (+)= sum_k S_g[(i,m_o), k] A_g[k, w]
//       sobek_gemm_sbar  Sbar_g[(i,m_o), k] = sum_w mbar(i, m_o, w) A_g[k, w]
//       sobek_gemm_ga    P[split, k, w]   = sum_{(i,m_o) in split} S_g[(i,m_o), k] mbar(i, m_o, w)
//     A_g[k, w] is read in place from W: row k of group g lives at W + ktab[k]
//     (ktab[k] = q*N_w + off_pi + u*C_out for k = koff_pi + q*C_in + u).
//   * sobek_ga_reduce: fixed-order sum of the split partials into W's layout.
//   * sobek_sender_reduce: deterministic x-gradient gather over the sender-sorted
//     view (Section 4.3: one fixed reduction order per source row).
//   * layout transposes (ir_mul <-> mul_ir, Section 4.5) and a column fill.
//
// MFMA 16x16x4 fp32 operand layout (lane l of the wave):
//   A[i][k] in lane i + 16k,  B[k][j] in lane j + 16k,
//   D[4g + r][j] in accumulator register r of lane j + 16g.

typedef float sb_f4 __attribute__((ext_vector_type(4)));
typedef long long sb_i64;

#define SB_DEV __device__ __forceinline__

SB_DEV sb_f4 sb_mfma(float a, float b, sb_f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// GEMM tiles: 256 threads = 4 waves; block tile BM=64 rows x BN columns, BK=16.
// Wave w owns rows [16w, 16w+16) and all BN columns (BN/16 MFMA tiles).
// ---------------------------------------------------------------------------
#define SB_BM 64
#define SB_BK 16

// out row r of group g -> address of (receiver r0 + r / dg, component r % dg) block.
SB_DEV sb_i64 sb_row_addr(int r, int dg, int Cg, int off, int CX, int r0) {
  return (sb_i64)(r0 + r / dg) * CX + off + (r % dg) * Cg;
}

template <int BN>
SB_DEV void sb_gemm_sa(const float* __restrict__ S, int nrows, int D, const float* __restrict__ W,
                       const int* __restrict__ ktab, float* __restrict__ out, int dg, int Cg, int off,
                       int CX, int r0, int accumulate) {
  __shared__ float sA[SB_BK][SB_BM + 4];
  __shared__ float sB[SB_BK][BN + 4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int rb = blockIdx.x * SB_BM, cb = blockIdx.y * BN;
  sb_f4 acc[BN / 16];
#pragma unroll
  for (int t = 0; t < BN / 16; ++t) acc[t] = (sb_f4){0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < D; k0 += SB_BK) {
    for (int idx = tid; idx < SB_BM * SB_BK; idx += 256) {
      int row = idx / SB_BK, kk = idx % SB_BK;
      int gr = rb + row, gk = k0 + kk;
      sA[kk][row] = (gr < nrows && gk < D) ? S[(sb_i64)gr * D + gk] : 0.f;
    }
    for (int idx = tid; idx < SB_BK * BN; idx += 256) {
      int kk = idx / BN, c = idx % BN;
      int gk = k0 + kk, gc = cb + c;
      sB[kk][c] = (gk < D && gc < Cg) ? W[(sb_i64)ktab[gk] + gc] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < SB_BK; kk += 4) {
      float a = sA[kk + (lane >> 4)][16 * wave + (lane & 15)];
#pragma unroll
      for (int t = 0; t < BN / 16; ++t) acc[t] = sb_mfma(a, sB[kk + (lane >> 4)][16 * t + (lane & 15)], acc[t]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int t = 0; t < BN / 16; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      int row = rb + 16 * wave + 4 * (lane >> 4) + r;
      int col = cb + 16 * t + (lane & 15);
      if (row < nrows && col < Cg) {
        float* o = out + sb_row_addr(row, dg, Cg, off, CX, r0) + col;
        *o = accumulate ? (*o + acc[t][r]) : acc[t][r];
      }
    }
}

template <int BN>
SB_DEV void sb_gemm_sbar(const float* __restrict__ M, int nrows, int D, const float* __restrict__ W,
                         const int* __restrict__ ktab, float* __restrict__ Sbar, int dg, int Cg, int off,
                         int CX, int r0) {
  __shared__ float sA[SB_BK][SB_BM + 4];
  __shared__ float sB[SB_BK][BN + 4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int rb = blockIdx.x * SB_BM, kb = blockIdx.y * BN;
  sb_f4 acc[BN / 16];
#pragma unroll
  for (int t = 0; t < BN / 16; ++t) acc[t] = (sb_f4){0.f, 0.f, 0.f, 0.f};
  for (int w0 = 0; w0 < Cg; w0 += SB_BK) {
    for (int idx = tid; idx < SB_BM * SB_BK; idx += 256) {
      int row = idx / SB_BK, ww = idx % SB_BK;
      int gr = rb + row, gw = w0 + ww;
      sA[ww][row] = (gr < nrows && gw < Cg) ? M[sb_row_addr(gr, dg, Cg, off, CX, r0) + gw] : 0.f;
    }
    for (int idx = tid; idx < SB_BK * BN; idx += 256) {
      int kc = idx / SB_BK, ww = idx % SB_BK;
      int gk = kb + kc, gw = w0 + ww;
      sB[ww][kc] = (gk < D && gw < Cg) ? W[(sb_i64)ktab[gk] + gw] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < SB_BK; kk += 4) {
      float a = sA[kk + (lane >> 4)][16 * wave + (lane & 15)];
#pragma unroll
      for (int t = 0; t < BN / 16; ++t) acc[t] = sb_mfma(a, sB[kk + (lane >> 4)][16 * t + (lane & 15)], acc[t]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int t = 0; t < BN / 16; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      int row = rb + 16 * wave + 4 * (lane >> 4) + r;
      int col = kb + 16 * t + (lane & 15);
      if (row < nrows && col < D) Sbar[(sb_i64)row * D + col] = acc[t][r];
    }
}

template <int BN>
SB_DEV void sb_gemm_ga(const float* __restrict__ S, int nrows, int D, const float* __restrict__ M,
                       float* __restrict__ P, int dg, int Cg, int off, int CX, int r0, int rows_per_split,
                       int accumulate) {
  __shared__ float sA[SB_BK][SB_BM + 4];
  __shared__ float sB[SB_BK][BN + 4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int kb = blockIdx.x * SB_BM, cb = blockIdx.y * BN, split = blockIdx.z;
  const int rbeg = split * rows_per_split;
  const int rend = min(nrows, rbeg + rows_per_split);
  sb_f4 acc[BN / 16];
#pragma unroll
  for (int t = 0; t < BN / 16; ++t) acc[t] = (sb_f4){0.f, 0.f, 0.f, 0.f};
  for (int r0b = rbeg; r0b < rend; r0b += SB_BK) {
    for (int idx = tid; idx < SB_BK * SB_BM; idx += 256) {
      int rr = idx / SB_BM, kk = idx % SB_BM;
      int gr = r0b + rr, gk = kb + kk;
      sA[rr][kk] = (gr < rend && gk < D) ? S[(sb_i64)gr * D + gk] : 0.f;
    }
    for (int idx = tid; idx < SB_BK * BN; idx += 256) {
      int rr = idx / BN, c = idx % BN;
      int gr = r0b + rr, gc = cb + c;
      sB[rr][c] = (gr < rend && gc < Cg) ? M[sb_row_addr(gr, dg, Cg, off, CX, r0) + gc] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < SB_BK; kk += 4) {
      float a = sA[kk + (lane >> 4)][16 * wave + (lane & 15)];
#pragma unroll
      for (int t = 0; t < BN / 16; ++t) acc[t] = sb_mfma(a, sB[kk + (lane >> 4)][16 * t + (lane & 15)], acc[t]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int t = 0; t < BN / 16; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      int k = kb + 16 * wave + 4 * (lane >> 4) + r;
      int col = cb + 16 * t + (lane & 15);
      if (k < D && col < Cg) {
        float* o = P + ((sb_i64)split * D + k) * Cg + col;
        *o = accumulate ? (*o + acc[t][r]) : acc[t][r];
      }
    }
}

#define SB_GEMM_ENTRY(BN)                                                                           \
  extern "C" __global__ __launch_bounds__(256) void sobek_gemm_sa_##BN(                            \
      const float* S, int nrows, int D, const float* W, const int* ktab, float* out, int dg,       \
      int Cg, int off, int CX, int r0, int accumulate) {                                           \
    sb_gemm_sa<BN>(S, nrows, D, W, ktab, out, dg, Cg, off, CX, r0, accumulate);                    \
  }                                                                                                \
  extern "C" __global__ __launch_bounds__(256) void sobek_gemm_sbar_##BN(                          \
      const float* M, int nrows, int D, const float* W, const int* ktab, float* Sbar, int dg,      \
      int Cg, int off, int CX, int r0) {                                                           \
    sb_gemm_sbar<BN>(M, nrows, D, W, ktab, Sbar, dg, Cg, off, CX, r0);                             \
  }                                                                                                \
  extern "C" __global__ __launch_bounds__(256) void sobek_gemm_ga_##BN(                            \
      const float* S, int nrows, int D, const float* M, float* P, int dg, int Cg, int off, int CX, \
      int r0, int rows_per_split, int accumulate) {                                                \
    sb_gemm_ga<BN>(S, nrows, D, M, P, dg, Cg, off, CX, r0, rows_per_split, accumulate);            \
  }

SB_GEMM_ENTRY(16)
SB_GEMM_ENTRY(32)
SB_GEMM_ENTRY(64)

// ---------------------------------------------------------------------------
// Vectorised channel GEMMs (every multiplicity a multiple of 4, so rows of S,
// W and the node tensors are 16-byte aligned): 128-row tiles (4 waves x 32
// rows), BK = 32, float4 global loads, and the next tile prefetched into
// registers while the MFMAs consume the current one from LDS.
// ---------------------------------------------------------------------------
#define SB_VM 128
#define SB_VK 32

typedef float sb_v4 __attribute__((ext_vector_type(4)));

SB_DEV sb_v4 sb_ld4(const float* p) { return *(const sb_v4*)p; }

// out rows (r0 + r / dg, r % dg) (+)= S[r, :] A_g, S row-major with row length D
template <int BN>
SB_DEV void sb_gemm_sa_v(const float* __restrict__ S, int nrows, int D, const float* __restrict__ W,
                         const int* __restrict__ ktab, float* __restrict__ out, int dg, int Cg, int off, int CX,
                         int r0, int accumulate, float* __restrict__ P, int kper) {
  __shared__ float sA[SB_VK][SB_VM + 4];
  __shared__ float sB[SB_VK][BN + 4];
  constexpr int NB = (SB_VK * BN / 4 + 255) / 256;  // float4 loads of B per thread
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int rb = blockIdx.x * SB_VM, cb = blockIdx.y * BN;
  // split z of a split-K launch takes k in [kbeg, kend) (kper a multiple of SB_VK)
  const int kbeg = blockIdx.z * kper, kend = min(D, kbeg + kper);
  sb_f4 acc[2][BN / 16];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int t = 0; t < BN / 16; ++t) acc[i][t] = (sb_f4){0.f, 0.f, 0.f, 0.f};
  sb_v4 ra[4], rbv[NB];
  auto load = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = (tid >> 3) + 32 * i, k = k0 + 4 * (tid & 7);
      const int gr = rb + row;
      ra[i] = (gr < nrows && k < kend) ? sb_ld4(S + (sb_i64)gr * D + k) : (sb_v4){0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int idx = tid + 256 * i;
      const int kk = idx / (BN / 4), c = 4 * (idx % (BN / 4));
      const int gk = k0 + kk;
      rbv[i] = (idx < SB_VK * BN / 4 && gk < kend && cb + c < Cg) ? sb_ld4(W + (sb_i64)ktab[gk] + cb + c)
                                                                : (sb_v4){0.f, 0.f, 0.f, 0.f};
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = (tid >> 3) + 32 * i, kq = 4 * (tid & 7);
#pragma unroll
      for (int c = 0; c < 4; ++c) sA[kq + c][row] = ra[i][c];
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int idx = tid + 256 * i;
      if (idx < SB_VK * BN / 4) *(sb_v4*)&sB[idx / (BN / 4)][4 * (idx % (BN / 4))] = rbv[i];
    }
  };
  load(kbeg);
  store();
  __syncthreads();
  for (int k0 = kbeg; k0 < kend; k0 += SB_VK) {
    const bool more = k0 + SB_VK < kend;
    if (more) load(k0 + SB_VK);
#pragma unroll
    for (int kk = 0; kk < SB_VK; kk += 4) {
      const float a0 = sA[kk + (lane >> 4)][32 * wave + (lane & 15)];
      const float a1 = sA[kk + (lane >> 4)][32 * wave + 16 + (lane & 15)];
#pragma unroll
      for (int t = 0; t < BN / 16; ++t) {
        const float b = sB[kk + (lane >> 4)][16 * t + (lane & 15)];
        acc[0][t] = sb_mfma(a0, b, acc[0][t]);
        acc[1][t] = sb_mfma(a1, b, acc[1][t]);
      }
    }
    __syncthreads();
    if (more) {
      store();
      __syncthreads();
    }
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int t = 0; t < BN / 16; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rb + 32 * wave + 16 * i + 4 * (lane >> 4) + r;
        const int col = cb + 16 * t + (lane & 15);
        if (row < nrows && col < Cg) {
          if (gridDim.z > 1) {  // partial of this split: P[z][row][col], summed by sobek_sa_reduce
            P[((sb_i64)blockIdx.z * nrows + row) * Cg + col] = acc[i][t][r];
          } else {
            float* o = out + sb_row_addr(row, dg, Cg, off, CX, r0) + col;
            *o = accumulate ? (*o + acc[i][t][r]) : acc[i][t][r];
          }
        }
      }
}

// out rows (r0 + r / dg, r % dg) (+)= sum_{z < nsplit} P[z][r][:], splits added in order
extern "C" __global__ __launch_bounds__(256) void sobek_sa_reduce(const float* __restrict__ P, int nsplit, int nrows,
                                                                  int Cg, float* __restrict__ out, int dg, int off,
                                                                  int CX, int r0, int accumulate) {
  const int nq = Cg / 4;
  const sb_i64 t = (sb_i64)blockIdx.x * 256 + threadIdx.x;
  if (t >= (sb_i64)nrows * nq) return;
  const int row = (int)(t / nq), c = 4 * (int)(t % nq);
  const sb_i64 stride = (sb_i64)nrows * Cg;
  const float* src = P + (sb_i64)row * Cg + c;
  sb_v4 v = sb_ld4(src);
  for (int z = 1; z < nsplit; ++z) v += sb_ld4(src + z * stride);
  sb_v4* o = (sb_v4*)(out + sb_row_addr(row, dg, Cg, off, CX, r0) + c);
  *o = accumulate ? (*o + v) : v;
}

// Sbar[r, k] = sum_w mbar(r, w) A_g[k, w]; 128 rows x 64 k-columns per block, reduction over w
SB_DEV void sb_gemm_sbar_v(const float* __restrict__ M, int nrows, int D, const float* __restrict__ W,
                           const int* __restrict__ ktab, float* __restrict__ Sbar, int dg, int Cg, int off, int CX,
                           int r0) {
  constexpr int BN = 64;
  __shared__ float sA[SB_VK][SB_VM + 4];
  __shared__ float sB[SB_VK][BN + 4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int rb = blockIdx.x * SB_VM, kb = blockIdx.y * BN;
  sb_f4 acc[2][BN / 16];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int t = 0; t < BN / 16; ++t) acc[i][t] = (sb_f4){0.f, 0.f, 0.f, 0.f};
  sb_v4 ra[4], rbv[2];
  auto load = [&](int w0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = (tid >> 3) + 32 * i, w = w0 + 4 * (tid & 7);
      const int gr = rb + row;
      ra[i] = (gr < nrows && w < Cg) ? sb_ld4(M + sb_row_addr(gr, dg, Cg, off, CX, r0) + w)
                                     : (sb_v4){0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int kc = (tid >> 3) + 32 * i, w = w0 + 4 * (tid & 7);
      const int gk = kb + kc;
      rbv[i] = (gk < D && w < Cg) ? sb_ld4(W + (sb_i64)ktab[gk] + w) : (sb_v4){0.f, 0.f, 0.f, 0.f};
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = (tid >> 3) + 32 * i, wq = 4 * (tid & 7);
#pragma unroll
      for (int c = 0; c < 4; ++c) sA[wq + c][row] = ra[i][c];
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int kc = (tid >> 3) + 32 * i, wq = 4 * (tid & 7);
#pragma unroll
      for (int c = 0; c < 4; ++c) sB[wq + c][kc] = rbv[i][c];
    }
  };
  load(0);
  store();
  __syncthreads();
  for (int w0 = 0; w0 < Cg; w0 += SB_VK) {
    const bool more = w0 + SB_VK < Cg;
    if (more) load(w0 + SB_VK);
#pragma unroll
    for (int kk = 0; kk < SB_VK; kk += 4) {
      const float a0 = sA[kk + (lane >> 4)][32 * wave + (lane & 15)];
      const float a1 = sA[kk + (lane >> 4)][32 * wave + 16 + (lane & 15)];
#pragma unroll
      for (int t = 0; t < BN / 16; ++t) {
        const float b = sB[kk + (lane >> 4)][16 * t + (lane & 15)];
        acc[0][t] = sb_mfma(a0, b, acc[0][t]);
        acc[1][t] = sb_mfma(a1, b, acc[1][t]);
      }
    }
    __syncthreads();
    if (more) {
      store();
      __syncthreads();
    }
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int t = 0; t < BN / 16; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rb + 32 * wave + 16 * i + 4 * (lane >> 4) + r;
        const int col = kb + 16 * t + (lane & 15);
        if (row < nrows && col < D) Sbar[(sb_i64)row * D + col] = acc[i][t][r];
      }
}

// Sbar[r, k] = sum_w mbar(r, w) A_g[k, w], streaming: a block owns 64 rows and
// walks all D columns in 64-column tiles.  Its mbar rows stay in LDS (transposed,
// [w][row]); A_g is consumed in slices of 64 columns x 32 w, the next slice loaded
// into registers while the current one is multiplied and then swapped into the
// other LDS buffer, so the block never waits on memory between slices and its LDS
// does not grow past one 32-wide slice pair with the multiplicity.  The product is
// taken transposed, Sbar^T tile = A_g tile x mbar^T (16x16x4 MFMA, A rows = k,
// B columns = rows), which leaves lane (j + 16 g) with columns 4g .. 4g + 3 of row
// j: one float4 store per 16x16 tile and lane.  CG (the group's multiplicity) is a
// multiple of 4; multiples of 16 take sb_gemm_sbar_w below.
template <int CG>
SB_DEV void sb_gemm_sbar_w(const float* __restrict__ M, int nrows, int D, const float* __restrict__ W,
                           const int* __restrict__ ktab, float* __restrict__ Sbar, int dg, int off, int CX, int r0);

template <int CG>
SB_DEV void sb_gemm_sbar_s(const float* __restrict__ M, int nrows, int D, const float* __restrict__ W,
                           const int* __restrict__ ktab, float* __restrict__ Sbar, int dg, int off, int CX, int r0) {
  if constexpr (CG % 16 == 0) {
    sb_gemm_sbar_w<CG>(M, nrows, D, W, ktab, Sbar, dg, off, CX, r0);
    return;
  }
  constexpr int PAD = 68;                       // row pitch of the transposed LDS tiles (floats)
  constexpr int NV = CG / 4;                    // float4 per row of mbar
  constexpr int WC = CG < 32 ? CG : 32;         // w per slice
  constexpr int NS = (CG + WC - 1) / WC;        // slices per column tile
  constexpr int NBL = (64 * (WC / 4) + 255) / 256;  // float4 loads of a slice per thread
  __shared__ float sM[CG][PAD];
  __shared__ float sB[2][WC][PAD];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int j = lane & 15, g = lane >> 4;
  const int rb = blockIdx.x * 64;
  for (int idx = tid; idx < 64 * NV; idx += 256) {
    const int row = idx / NV, w4 = 4 * (idx % NV);
    const int gr = rb + row;
    const sb_v4 v = gr < nrows ? sb_ld4(M + sb_row_addr(gr, dg, CG, off, CX, r0) + w4) : (sb_v4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < 4; ++c) sM[w4 + c][row] = v[c];
  }
  sb_v4 rbv[NBL];
  auto loadB = [&](int sl) {  // slice sl = (column tile, w chunk)
    const int k0 = (sl / NS) * 64, w0 = (sl % NS) * WC;
#pragma unroll
    for (int i = 0; i < NBL; ++i) {
      const int idx = tid + 256 * i;
      const int kc = idx / (WC / 4), w4 = 4 * (idx % (WC / 4)), gk = k0 + kc;
      rbv[i] = (idx < 64 * (WC / 4) && gk < D && w0 + w4 < CG) ? sb_ld4(W + (sb_i64)ktab[gk] + w0 + w4)
                                                                 : (sb_v4){0.f, 0.f, 0.f, 0.f};
    }
  };
  auto storeB = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NBL; ++i) {
      const int idx = tid + 256 * i;
      if (idx < 64 * (WC / 4)) {
        const int kc = idx / (WC / 4), w4 = 4 * (idx % (WC / 4));
#pragma unroll
        for (int c = 0; c < 4; ++c) sB[buf][w4 + c][kc] = rbv[i][c];
      }
    }
  };
  // blockIdx.y takes a contiguous range of 64-wide column tiles
  const int ntile = (D + 63) / 64, tpb = (ntile + gridDim.y - 1) / gridDim.y;
  const int sl0 = blockIdx.y * tpb * NS, nsl = min(ntile, (int)(blockIdx.y + 1) * tpb) * NS;
  loadB(sl0);
  storeB(0);
  __syncthreads();
  const int row = rb + 16 * wave + j;
  float* out = Sbar + (sb_i64)row * D;
  sb_f4 acc[4];
  for (int sl = sl0; sl < nsl; ++sl) {
    const int buf = (sl - sl0) & 1, w0 = (sl % NS) * WC;
    if (sl + 1 < nsl) loadB(sl + 1);
    if (w0 == 0) {
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[t] = (sb_f4){0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int w = 0; w < WC; w += 4) {
      const float b = sM[w0 + w + g][16 * wave + j];
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[t] = sb_mfma(sB[buf][w + g][16 * t + j], b, acc[t]);
    }
    if (w0 + WC >= CG && row < nrows) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int k = (sl / NS) * 64 + 16 * t + 4 * g;
        if (k < D) *(sb_v4*)(out + k) = acc[t];
      }
    }
    if (sl + 1 < nsl) storeB(buf ^ 1);
    __syncthreads();
  }
}

// The streaming Sbar GEMM for multiplicities in multiples of 16, with w-contiguous LDS rows: the
// block's mbar rows as stored ([row][w], pitch CG + 4 floats) and A's slice as [k][w] (pitch WC + 4),
// so a lane takes four consecutive w of its A row and of its mbar row with one 16-byte LDS read each
// (the row pitches keep eight lanes' reads on distinct banks).  The 16x16x4 MFMA sums over its four
// lane groups; in step s of a 16-wide block of w, lane group g supplies w = 4g + s for both operands,
// so four steps cover the block.  Blocking, slices, the column-tile split and the stores are those of
// sb_gemm_sbar_s.
template <int CG>
SB_DEV void sb_gemm_sbar_w(const float* __restrict__ M, int nrows, int D, const float* __restrict__ W,
                           const int* __restrict__ ktab, float* __restrict__ Sbar, int dg, int off, int CX, int r0) {
  static_assert(CG % 16 == 0, "16-wide blocks of w");
  constexpr int WC = CG < 32 ? CG : 32;         // w per slice (16 or 32; divides CG)
  constexpr int NS = CG / WC;                   // slices per column tile
  constexpr int PM = CG + 4, PB = WC + 4;       // LDS row pitches (floats)
  constexpr int NV = CG / 4;                    // float4 per row of mbar
  constexpr int NBL = (64 * (WC / 4) + 255) / 256;  // float4 loads of a slice per thread
  __shared__ __attribute__((aligned(16))) float sM[64 * PM];
  __shared__ __attribute__((aligned(16))) float sB[2][64 * PB];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int j = lane & 15, g = lane >> 4;
  const int rb = blockIdx.x * 64;
  for (int idx = tid; idx < 64 * NV; idx += 256) {
    const int row = idx / NV, w4 = 4 * (idx % NV);
    const int gr = rb + row;
    *(sb_v4*)&sM[row * PM + w4] =
        gr < nrows ? sb_ld4(M + sb_row_addr(gr, dg, CG, off, CX, r0) + w4) : (sb_v4){0.f, 0.f, 0.f, 0.f};
  }
  sb_v4 rbv[NBL];
  auto loadB = [&](int sl) {  // slice sl = (column tile, w chunk)
    const int k0 = (sl / NS) * 64, w0 = (sl % NS) * WC;
#pragma unroll
    for (int i = 0; i < NBL; ++i) {
      const int idx = tid + 256 * i;
      const int kc = idx / (WC / 4), w4 = 4 * (idx % (WC / 4)), gk = k0 + kc;
      rbv[i] = (idx < 64 * (WC / 4) && gk < D) ? sb_ld4(W + (sb_i64)ktab[gk] + w0 + w4) : (sb_v4){0.f, 0.f, 0.f, 0.f};
    }
  };
  auto storeB = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NBL; ++i) {
      const int idx = tid + 256 * i;
      if (idx < 64 * (WC / 4)) *(sb_v4*)&sB[buf][(idx / (WC / 4)) * PB + 4 * (idx % (WC / 4))] = rbv[i];
    }
  };
  // blockIdx.y takes a contiguous range of 64-wide column tiles
  const int ntile = (D + 63) / 64, tpb = (ntile + gridDim.y - 1) / gridDim.y;
  const int sl0 = blockIdx.y * tpb * NS, nsl = min(ntile, (int)(blockIdx.y + 1) * tpb) * NS;
  loadB(sl0);
  storeB(0);
  __syncthreads();
  const int row = rb + 16 * wave + j;
  float* out = Sbar + (sb_i64)row * D;
  const float* mrow = &sM[(16 * wave + j) * PM + 4 * g];
  sb_f4 acc[4];
  for (int sl = sl0; sl < nsl; ++sl) {
    const int buf = (sl - sl0) & 1, w0 = (sl % NS) * WC;
    if (sl + 1 < nsl) loadB(sl + 1);
    if (w0 == 0) {
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[t] = (sb_f4){0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int wb = 0; wb < WC; wb += 16) {
      const sb_v4 b = *(const sb_v4*)(mrow + w0 + wb);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const sb_v4 a = *(const sb_v4*)&sB[buf][(16 * t + j) * PB + wb + 4 * g];
#pragma unroll
        for (int s = 0; s < 4; ++s) acc[t] = sb_mfma(a[s], b[s], acc[t]);
      }
    }
    if (w0 + WC >= CG && row < nrows) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int k = (sl / NS) * 64 + 16 * t + 4 * g;
        if (k < D) *(sb_v4*)(out + k) = acc[t];
      }
    }
    if (sl + 1 < nsl) storeB(buf ^ 1);
    __syncthreads();
  }
}

// P[split, k, w] = sum_{r in split} S[r, k] mbar(r, w); 128 k-rows x BN columns per block
template <int BN>
SB_DEV void sb_gemm_ga_v(const float* __restrict__ S, int nrows, int D, const float* __restrict__ M,
                         float* __restrict__ P, int dg, int Cg, int off, int CX, int r0, int rows_per_split,
                         int accumulate) {
  __shared__ float sA[SB_VK][SB_VM + 4];
  __shared__ float sB[SB_VK][BN + 4];
  constexpr int NB = (SB_VK * BN / 4 + 255) / 256;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int kb = blockIdx.x * SB_VM, cb = blockIdx.y * BN, split = blockIdx.z;
  const int rbeg = split * rows_per_split;
  const int rend = min(nrows, rbeg + rows_per_split);
  sb_f4 acc[2][BN / 16];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int t = 0; t < BN / 16; ++t) acc[i][t] = (sb_f4){0.f, 0.f, 0.f, 0.f};
  sb_v4 ra[4], rbv[NB];
  auto load = [&](int rr0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rr = (tid >> 5) + 8 * i, k = kb + 4 * (tid & 31);
      const int gr = rr0 + rr;
      ra[i] = (gr < rend && k < D) ? sb_ld4(S + (sb_i64)gr * D + k) : (sb_v4){0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int idx = tid + 256 * i;
      const int rr = idx / (BN / 4), c = 4 * (idx % (BN / 4));
      const int gr = rr0 + rr;
      rbv[i] = (idx < SB_VK * BN / 4 && gr < rend && cb + c < Cg)
                   ? sb_ld4(M + sb_row_addr(gr, dg, Cg, off, CX, r0) + cb + c)
                   : (sb_v4){0.f, 0.f, 0.f, 0.f};
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rr = (tid >> 5) + 8 * i;
      *(sb_v4*)&sA[rr][4 * (tid & 31)] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int idx = tid + 256 * i;
      if (idx < SB_VK * BN / 4) *(sb_v4*)&sB[idx / (BN / 4)][4 * (idx % (BN / 4))] = rbv[i];
    }
  };
  if (rbeg < rend) {
    load(rbeg);
    store();
  }
  __syncthreads();
  for (int rr0 = rbeg; rr0 < rend; rr0 += SB_VK) {
    const bool more = rr0 + SB_VK < rend;
    if (more) load(rr0 + SB_VK);
#pragma unroll
    for (int kk = 0; kk < SB_VK; kk += 4) {
      const float a0 = sA[kk + (lane >> 4)][32 * wave + (lane & 15)];
      const float a1 = sA[kk + (lane >> 4)][32 * wave + 16 + (lane & 15)];
#pragma unroll
      for (int t = 0; t < BN / 16; ++t) {
        const float b = sB[kk + (lane >> 4)][16 * t + (lane & 15)];
        acc[0][t] = sb_mfma(a0, b, acc[0][t]);
        acc[1][t] = sb_mfma(a1, b, acc[1][t]);
      }
    }
    __syncthreads();
    if (more) {
      store();
      __syncthreads();
    }
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int t = 0; t < BN / 16; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int k = kb + 32 * wave + 16 * i + 4 * (lane >> 4) + r;
        const int col = cb + 16 * t + (lane & 15);
        if (k < D && col < Cg) {
          float* o = P + ((sb_i64)split * D + k) * Cg + col;
          *o = accumulate ? (*o + acc[i][t][r]) : acc[i][t][r];
        }
      }
}

#define SB_GEMM_V_ENTRY(BN)                                                                          \
  extern "C" __global__ __launch_bounds__(256) void sobek_gemm_sa_v##BN(                            \
      const float* S, int nrows, int D, const float* W, const int* ktab, float* out, int dg,       \
      int Cg, int off, int CX, int r0, int accumulate, float* P, int kper) {                       \
    sb_gemm_sa_v<BN>(S, nrows, D, W, ktab, out, dg, Cg, off, CX, r0, accumulate, P, kper);         \
  }                                                                                                \
  extern "C" __global__ __launch_bounds__(256) void sobek_gemm_ga_v##BN(                            \
      const float* S, int nrows, int D, const float* M, float* P, int dg, int Cg, int off, int CX, \
      int r0, int rows_per_split, int accumulate) {                                                \
    sb_gemm_ga_v<BN>(S, nrows, D, M, P, dg, Cg, off, CX, r0, rows_per_split, accumulate);          \
  }

SB_GEMM_V_ENTRY(16)
SB_GEMM_V_ENTRY(32)
SB_GEMM_V_ENTRY(64)

extern "C" __global__ __launch_bounds__(256) void sobek_gemm_sbar_v(const float* M, int nrows, int D, const float* W,
                                                                    const int* ktab, float* Sbar, int dg, int Cg,
                                                                    int off, int CX, int r0) {
  sb_gemm_sbar_v(M, nrows, D, W, ktab, Sbar, dg, Cg, off, CX, r0);
}

// ---------------------------------------------------------------------------
// Channelwise (uvu) mixing, eq. uvu_connection in receiver form: a path's
// weights A[q, path, u] pair state column k = koff + q*C + u with output
// channel u only, so the three channel products are elementwise in u and
// reduce over (path, q) or over rows; ktab[k] is the W offset of column k.
// Memory bound: one pass over the state (or its adjoint) per launch.
// ---------------------------------------------------------------------------

// out rows (r0 + r / dg, r % dg), channel u (+)= sum_j W[ktab[j*C + u]] S[r, j*C + u]
extern "C" __global__ __launch_bounds__(256) void sobek_uvu_mix(const float* __restrict__ S, int nrows, int D, int C,
                                                                const float* __restrict__ W,
                                                                const int* __restrict__ ktab, float* __restrict__ out,
                                                                int dg, int off, int CX, int r0, int accumulate) {
  const sb_i64 t = (sb_i64)blockIdx.x * 256 + threadIdx.x;
  if (t >= (sb_i64)nrows * C) return;
  const int r = (int)(t / C), u = (int)(t % C);
  const float* s = S + (sb_i64)r * D + u;
  float acc = 0.f;
  for (int k = 0; k < D; k += C) acc += W[ktab[k + u]] * s[k];
  float* o = out + sb_row_addr(r, dg, C, off, CX, r0) + u;
  *o = accumulate ? (*o + acc) : acc;
}

// Sbar[r, k] = mbar(row r, channel k % C) W[ktab[k]]
extern "C" __global__ __launch_bounds__(256) void sobek_uvu_sbar(const float* __restrict__ M, int nrows, int D, int C,
                                                                 const float* __restrict__ W,
                                                                 const int* __restrict__ ktab,
                                                                 float* __restrict__ Sbar, int dg, int off, int CX,
                                                                 int r0) {
  const sb_i64 t = (sb_i64)blockIdx.x * 256 + threadIdx.x;
  if (t >= (sb_i64)nrows * D) return;
  const int r = (int)(t / D), k = (int)(t % D);
  Sbar[t] = M[sb_row_addr(r, dg, C, off, CX, r0) + k % C] * W[ktab[k]];
}

// P[split, k] (+)= sum over the split's rows r of S[r, k] mbar(row r, channel k % C)
extern "C" __global__ __launch_bounds__(256) void sobek_uvu_ga(const float* __restrict__ S, int nrows, int D, int C,
                                                               const float* __restrict__ M, float* __restrict__ P,
                                                               int dg, int off, int CX, int r0, int rows_per_split,
                                                               int accumulate) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  if (k >= D) return;
  const int rbeg = blockIdx.z * rows_per_split, rend = min(nrows, rbeg + rows_per_split);
  const int u = k % C;
  float acc = 0.f;
  for (int r = rbeg; r < rend; ++r) acc += S[(sb_i64)r * D + k] * M[sb_row_addr(r, dg, C, off, CX, r0) + u];
  float* o = P + (sb_i64)blockIdx.z * D + k;
  *o = accumulate ? (*o + acc) : acc;
}

// gW[i] = sum over rows r < nrows of part[r][i], i < n, rows added in order
extern "C" __global__ __launch_bounds__(256) void sobek_uvu_wreduce(const float* __restrict__ part, int nrows,
                                                                    sb_i64 n, float* __restrict__ gW) {
  const sb_i64 i = (sb_i64)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  int r = 0;
  for (; r + 8 <= nrows; r += 8) {  // eight loads in flight, added in row order
    float v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = part[(sb_i64)(r + k) * n + i];
#pragma unroll
    for (int k = 0; k < 8; ++k) s += v[k];
  }
  for (; r < nrows; ++r) s += part[(sb_i64)r * n + i];
  gW[i] = s;
}

// gW[ktab[k] + w] = (first ? 0 : gW[..]) + sum_{s < nsplit} P[s, k, w]   (fixed split order)
extern "C" __global__ __launch_bounds__(256) void sobek_ga_reduce(const float* P, int nsplit, int D, int Cg,
                                                                  const int* ktab, float* gW, int first) {
  sb_i64 t = (sb_i64)blockIdx.x * 256 + threadIdx.x;
  if (t >= (sb_i64)D * Cg) return;
  int k = (int)(t / Cg), w = (int)(t % Cg);
  const sb_i64 stride = (sb_i64)D * Cg;
  const float* src = P + t;
  float s = 0.f;
  int p = 0;
  for (; p + 8 <= nsplit; p += 8) {  // eight loads in flight, added in split order
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = src[(p + i) * stride];
#pragma unroll
    for (int i = 0; i < 8; ++i) s += v[i];
  }
  for (; p < nsplit; ++p) s += src[p * stride];
  float* o = gW + (sb_i64)ktab[k] + w;
  *o = first ? s : (*o + s);
}

// One wave per sender j: x-gradient rows are the sum, in sender-CSR order, of the
// per-edge contribution rows of its out-edges inside the receiver chunk [e0, e1)
// (contributions are stored at row e - e0).  Chunks arrive in increasing edge
// order, so each sender's edges inside a chunk continue where the previous chunk
// stopped: cursor[j] keeps that position.  first: chunk 0 overwrites every row
// and initialises the cursors.
//
// The wave reads 64 sender-CSR slots at once (one per lane); the edge ids of
// the chunk are handed to the whole wave with readlane, and the rows of four
// edges are loaded before they are added (in edge order), so every lane keeps
// several row loads in flight.  Lane l owns the float4 columns l, l + 64, ... of
// the row (CX a multiple of 4) or the scalar columns l, l + 64, ... (otherwise).
template <int CX>
SB_DEV void sb_sender_reduce(const int* __restrict__ send_rowptr, const int* __restrict__ send_perm,
                             const float* __restrict__ contrib, float* __restrict__ gx, int* __restrict__ cursor,
                             int N, int e0, int e1, int first) {
  constexpr bool V4 = (CX % 4) == 0;
  constexpr int W = V4 ? 4 : 1;             // floats per lane access
  constexpr int NC = CX / W;                // accesses per row
  constexpr int R = (NC + 63) / 64;         // accesses per lane per row
  typedef float vt __attribute__((ext_vector_type(W)));
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (j >= N) return;
  const int start = first ? send_rowptr[j] : cursor[j];
  const int lim = send_rowptr[j + 1];
  vt acc[R];
#pragma unroll
  for (int r = 0; r < R; ++r) acc[r] = (vt)(0.f);
  auto row = [&](int e, int r) -> vt {
    const int c = lane + 64 * r;
    return c < NC ? *(const vt*)(contrib + (sb_i64)(e - e0) * CX + W * c) : (vt)(0.f);
  };
  int n = 0;
  for (;;) {
    // the chunk's edges of this sender form a prefix of [start, lim): perm is
    // increasing along a sender's slots
    const int p = start + n + lane;
    const int pe = p < lim ? send_perm[p] : 0x7fffffff;
    const int cnt = __popcll(__ballot(pe < e1));
    int t = 0;
    for (; t + 4 <= cnt; t += 4) {
      const int ea = __builtin_amdgcn_readlane(pe, t), eb = __builtin_amdgcn_readlane(pe, t + 1);
      const int ec = __builtin_amdgcn_readlane(pe, t + 2), ed = __builtin_amdgcn_readlane(pe, t + 3);
      vt va[R], vb[R], vc[R], vd[R];
#pragma unroll
      for (int r = 0; r < R; ++r) { va[r] = row(ea, r); vb[r] = row(eb, r); vc[r] = row(ec, r); vd[r] = row(ed, r); }
#pragma unroll
      for (int r = 0; r < R; ++r) acc[r] = (((acc[r] + va[r]) + vb[r]) + vc[r]) + vd[r];
    }
    for (; t < cnt; ++t) {
      const int ea = __builtin_amdgcn_readlane(pe, t);
#pragma unroll
      for (int r = 0; r < R; ++r) acc[r] += row(ea, r);
    }
    n += cnt;
    if (cnt < 64) break;
  }
  if (lane == 0) cursor[j] = start + n;
  if (!first && n == 0) return;
  float* out = gx + (sb_i64)j * CX;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int c = lane + 64 * r;
    if (c < NC) {
      vt* o = (vt*)(out + W * c);
      *o = first ? acc[r] : (*o + acc[r]);
    }
  }
}

// Layout transpose of one irrep block per launch row: for node n and block
// (off, C, d): ir_mul index off + m*C + u  <->  mul_ir index off + u*d + m.
// dir = 0: mul_ir -> ir_mul, dir = 1: ir_mul -> mul_ir.
extern "C" __global__ __launch_bounds__(256) void sobek_transpose(const float* src, float* dst, int N, int CX,
                                                                  const int* boff, const int* bmul,
                                                                  const int* bdim, int nblocks, int dir) {
  sb_i64 t = (sb_i64)blockIdx.x * 256 + threadIdx.x;
  if (t >= (sb_i64)N * CX) return;
  int n = (int)(t / CX), col = (int)(t % CX);
  int b = 0;
  while (b + 1 < nblocks && boff[b + 1] <= col) ++b;
  int C = bmul[b], d = bdim[b], r = col - boff[b];
  int m = r / C, u = r % C;  // col read as ir_mul (m, u)
  int other = boff[b] + u * d + m;
  if (dir == 0) dst[(sb_i64)n * CX + col] = src[(sb_i64)n * CX + other];
  else dst[(sb_i64)n * CX + other] = src[(sb_i64)n * CX + col];
}

// out[n][off + c] = 0 for c < width (output irreps no path reaches).
extern "C" __global__ __launch_bounds__(256) void sobek_fill_cols(float* out, int N, int CX, int off, int width) {
  sb_i64 t = (sb_i64)blockIdx.x * 256 + threadIdx.x;
  if (t >= (sb_i64)N * width) return;
  int n = (int)(t / width), c = (int)(t % width);
  out[(sb_i64)n * CX + off + c] = 0.f;
}

// Every value of buf[0..n) = 0 (used instead of memset so the stream stays capture-safe).
extern "C" __global__ __launch_bounds__(256) void sobek_zero(float* buf, sb_i64 n) {
  sb_i64 t = (sb_i64)blockIdx.x * 256 + threadIdx.x;
  if (t < n) buf[t] = 0.f;
}
