// The channel GEMMs on bf16 MFMA, for plans built with the dtype
// SOBEK_DTYPE_BF16_GEMM: m_g = S_g A_g (Section 4.2 eq. receiver_matrix_product),
// the weight gradient A_bar = S^T mbar and the adjoint state Sbar = mbar A^T
// (Section 4.3 eq. receiver_adjoint), which the paper runs as fp32 GEMMs.  The generator appends this file to the
// plan's source only for such plans; it relies on the fp32 device code that
// precedes every plan (sb_gemm_sa_v's tiling constants, loads and row mapping).
//
// Same blocking and staging as sb_gemm_sa_v: a 128-row x BN-column block, four
// waves of 32 rows, 32-deep k slabs of S and A staged in LDS as fp32 and the
// next slab prefetched into registers.  Each 16x16 tile then takes one
// v_mfma_f32_16x16x32_bf16 per slab instead of eight v_mfma_f32_16x16x4_f32:
// the lane's eight k values of S and of A are rounded to bf16 (round to nearest
// even, v_cvt_pk_bf16_f32) as they leave LDS, and products accumulate in fp32.
//
// Operand layout of v_mfma_f32_16x16x32_bf16 (lane l of the wave): A row
// (l & 15) and B column (l & 15) supply the eight k values of slot group
// l >> 4; both operands use the same slot for the same k, so the tile sums
// S[i][k] A[k][j] over the 32 k of the slab.  D[4g + r][j] sits in accumulator
// register r of lane j + 16g, as for the fp32 instruction.

typedef __bf16 sb_b8 __attribute__((ext_vector_type(8)));
typedef __bf16 sb_b4 __attribute__((ext_vector_type(4)));

// Four consecutive bf16 values of the receiver state (stored in bf16 by the state kernels of these
// plans), widened to fp32 for the LDS stage.
SB_DEV sb_v4 sb_ld4_b(const __bf16* p) {
  const sb_b4 v = *(const sb_b4*)p;
  return (sb_v4){(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
}

// acc += the 32-deep slab product of sA[kk][32 * wave + 0..31] and sB[kk][0..BN-1]
// (kk = 0..31, the reduction index), rounded to bf16 as it leaves LDS
template <int BN>
SB_DEV void sb_slab_bf16(const float (*sA)[SB_VM + 4], const float (*sB)[BN + 4], int wave, int lane,
                         sb_f4 (&acc)[2][BN / 16]) {
  const int kg = 8 * (lane >> 4), li = lane & 15;
  sb_b8 a0, a1;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    a0[j] = (__bf16)sA[kg + j][32 * wave + li];
    a1[j] = (__bf16)sA[kg + j][32 * wave + 16 + li];
  }
#pragma unroll
  for (int t = 0; t < BN / 16; ++t) {
    sb_b8 b;
#pragma unroll
    for (int j = 0; j < 8; ++j) b[j] = (__bf16)sB[kg + j][16 * t + li];
    acc[0][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b, acc[0][t], 0, 0, 0);
    acc[1][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b, acc[1][t], 0, 0, 0);
  }
}

template <int BN>
SB_DEV void sb_gemm_sa_vb(const __bf16* __restrict__ S, int nrows, int D, const float* __restrict__ W,
                          const int* __restrict__ ktab, float* __restrict__ out, int dg, int Cg, int off, int CX,
                          int r0, int accumulate, float* __restrict__ P, int kper) {
  __shared__ float sA[SB_VK][SB_VM + 4];
  __shared__ float sB[SB_VK][BN + 4];
  static_assert(SB_VK == 32, "one 32-deep bf16 MFMA per slab");
  constexpr int NB = (SB_VK * BN / 4 + 255) / 256;  // float4 loads of B per thread
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int rb = blockIdx.x * SB_VM, cb = blockIdx.y * BN;
  const int kbeg = blockIdx.z * kper, kend = min(D, kbeg + kper);
  const int li = lane & 15;
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
      ra[i] = (gr < nrows && k < kend) ? sb_ld4_b(S + (sb_i64)gr * D + k) : (sb_v4){0.f, 0.f, 0.f, 0.f};
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
    sb_slab_bf16<BN>(sA, sB, wave, lane, acc);
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
        const int col = cb + 16 * t + li;
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

// Weight-gradient partials P[split][k][w] (+)= sum over the split's rows r of S[r][k] mbar(r, w)
// (Section 4.3 eq. receiver_adjoint, A_bar = S^T mbar): the blocking of sb_gemm_ga_v (a 128-k x
// BN-w block walking 32-row slabs of its split), with the slab product on bf16 MFMA.
template <int BN>
SB_DEV void sb_gemm_ga_vb(const __bf16* __restrict__ S, int nrows, int D, const float* __restrict__ M,
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
      ra[i] = (gr < rend && k < D) ? sb_ld4_b(S + (sb_i64)gr * D + k) : (sb_v4){0.f, 0.f, 0.f, 0.f};
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
    sb_slab_bf16<BN>(sA, sB, wave, lane, acc);
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

#define SB_GEMM_VB_ENTRY(BN)                                                                         \
  extern "C" __global__ __launch_bounds__(256) void sobek_gemm_sa_vb##BN(                           \
      const __bf16* S, int nrows, int D, const float* W, const int* ktab, float* out, int dg,       \
      int Cg, int off, int CX, int r0, int accumulate, float* P, int kper) {                       \
    sb_gemm_sa_vb<BN>(S, nrows, D, W, ktab, out, dg, Cg, off, CX, r0, accumulate, P, kper);        \
  }                                                                                                \
  extern "C" __global__ __launch_bounds__(256) void sobek_gemm_ga_vb##BN(                           \
      const __bf16* S, int nrows, int D, const float* M, float* P, int dg, int Cg, int off, int CX, \
      int r0, int rows_per_split, int accumulate) {                                                \
    sb_gemm_ga_vb<BN>(S, nrows, D, M, P, dg, Cg, off, CX, r0, rows_per_split, accumulate);         \
  }

SB_GEMM_VB_ENTRY(16)
SB_GEMM_VB_ENTRY(32)
SB_GEMM_VB_ENTRY(64)
SB_GEMM_VB_ENTRY(128)  // groups over 64 channels: each block reads its rows of S once

// Adjoint state Sbar_g = mbar_g A_g^T (Section 4.3 eq. receiver_adjoint) on bf16 MFMA, streaming:
// a block owns SB_SBR rows of mbar (kept in LDS in bf16, w contiguous) and walks its range of 64-wide
// column tiles of Sbar in 32-deep slices of w, A's slice double-buffered in LDS (bf16, w contiguous).
// Wave v owns rows 64v .. 64v + 63 of the block (four 16-row tiles), so each slice costs sixteen
// v_mfma_f32_16x16x32_bf16 per wave, and A_g is read once per SB_SBR rows: the group's A (several MB
// for 128-channel groups, beyond one XCD's L2) would otherwise be streamed again for every 64 rows.
// Operands are rounded to bf16 (nearest even) as they enter LDS; products accumulate in fp32 and Sbar
// is written in fp32.  Lane (j + 16 g) supplies w = 8g .. 8g + 7 of its A row and mbar row, one 16-byte
// LDS read each; the product is taken transposed (rows of the tile = k), which leaves the lane with
// columns 4g .. 4g + 3 of row j: one float4 store per tile.  CG (the group's multiplicity) is a multiple
// of 32, at most 128 (the mbar rows then take at most 68 KB of LDS).
#define SB_SBR 256

template <int CG>
SB_DEV void sb_gemm_sbar_sb(const float* __restrict__ M, int nrows, int D, const float* __restrict__ W,
                            const int* __restrict__ ktab, float* __restrict__ Sbar, int dg, int off, int CX,
                            int r0) {
  static_assert(CG % 32 == 0 && CG <= 128, "32-deep slices of w, mbar rows within LDS");
  constexpr int WC = 32;                        // w per slice
  constexpr int NS = CG / WC;                   // slices per column tile
  constexpr int PM = CG + 8, PB = WC + 8;       // LDS row pitches (bf16)
  constexpr int NV = CG / 4;                    // float4 per row of mbar
  constexpr int NBL = (64 * (WC / 4) + 255) / 256;  // float4 loads of a slice per thread
  __shared__ __attribute__((aligned(16))) __bf16 sM[SB_SBR * PM];
  __shared__ __attribute__((aligned(16))) __bf16 sB[2][64 * PB];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int j = lane & 15, g = lane >> 4;
  const int rb = blockIdx.x * SB_SBR;
  auto put4 = [](__bf16* p, sb_v4 v) {  // four values rounded to bf16, one 8-byte LDS store
    *(sb_b4*)p = (sb_b4){(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
  };
  for (int idx = tid; idx < SB_SBR * NV; idx += 256) {
    const int row = idx / NV, w4 = 4 * (idx % NV);
    const int gr = rb + row;
    put4(&sM[row * PM + w4],
         gr < nrows ? sb_ld4(M + sb_row_addr(gr, dg, CG, off, CX, r0) + w4) : (sb_v4){0.f, 0.f, 0.f, 0.f});
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
      if (idx < 64 * (WC / 4)) put4(&sB[buf][(idx / (WC / 4)) * PB + 4 * (idx % (WC / 4))], rbv[i]);
    }
  };
  // blockIdx.y takes a contiguous range of 64-wide column tiles
  const int ntile = (D + 63) / 64, tpb = (ntile + gridDim.y - 1) / gridDim.y;
  const int sl0 = blockIdx.y * tpb * NS, nsl = min(ntile, (int)(blockIdx.y + 1) * tpb) * NS;
  loadB(sl0);
  storeB(0);
  __syncthreads();
  sb_f4 acc[4][4];  // [row tile][column tile]
  for (int sl = sl0; sl < nsl; ++sl) {
    const int buf = (sl - sl0) & 1, w0 = (sl % NS) * WC;
    if (sl + 1 < nsl) loadB(sl + 1);
    if (w0 == 0) {
#pragma unroll
      for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[rt][t] = (sb_f4){0.f, 0.f, 0.f, 0.f};
    }
    sb_b8 a[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) a[t] = *(const sb_b8*)&sB[buf][(16 * t + j) * PB + 8 * g];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
      const sb_b8 b = *(const sb_b8*)&sM[(64 * wave + 16 * rt + j) * PM + w0 + 8 * g];
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[rt][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[t], b, acc[rt][t], 0, 0, 0);
    }
    if (w0 + WC >= CG) {
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        const int row = rb + 64 * wave + 16 * rt + j;
        if (row < nrows) {
          float* out = Sbar + (sb_i64)row * D;
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const int k = (sl / NS) * 64 + 16 * t + 4 * g;
            if (k < D) *(sb_v4*)(out + k) = acc[rt][t];
          }
        }
      }
    }
    if (sl + 1 < nsl) storeB(buf ^ 1);
    __syncthreads();
  }
}
