// Device-side stand-ins for compiling generated HIP kernels for the host (CPU emulation).
#pragma once
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <cmath>
#include <tuple>
#include <type_traits>
#include <utility>

#include "emu_rt.h"

#ifdef EMU_SCAN
#define __global__ EMU_GLOBAL_MARK
#else
#define __global__
#endif
#define __device__
#define __host__
#define __forceinline__ inline
#define __shared__ static __attribute__((section("emu_lds")))
#define __launch_bounds__(...)
#define threadIdx (emu_cur->tid)
#define blockIdx emu_blockIdx
#define blockDim emu_blockDim
#define gridDim emu_gridDim
#define __syncthreads() emu_syncthreads(__LINE__)
#define __popcll(x) __builtin_popcountll(x)
#define __builtin_amdgcn_sched_barrier(x) ((void)0)
#define __builtin_amdgcn_fence(a, b) ((void)0)
#define __builtin_amdgcn_wave_barrier() emu_wave_sync(__LINE__)
#define __builtin_amdgcn_rsqf(x) (1.0f / sqrtf(x))
#define __builtin_amdgcn_readlane(v, l) emu_readlane((v), (l), __LINE__)
#define __ballot(p) emu_ballot((p), __LINE__)
#define __shfl_xor(...) emu_shfl_xor_(__LINE__, __VA_ARGS__)
#define __builtin_amdgcn_mfma_f32_4x4x1f32(a, b, c, x, y, z) emu_mfma_4x4x1((a), (b), (c), __LINE__)
#define __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, x, y, z) emu_mfma_16x16x4((a), (b), (c), __LINE__)
#define __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, x, y, z) emu_mfma_16x16x32_bf16((a), (b), (c), __LINE__)

template <class A, class B>
static inline std::common_type_t<A, B> min(A a, B b) { return b < a ? b : a; }
template <class A, class B>
static inline std::common_type_t<A, B> max(A a, B b) { return a < b ? b : a; }

typedef float emu_f4 __attribute__((ext_vector_type(4)));
typedef __bf16 emu_b8 __attribute__((ext_vector_type(8)));

static inline void emu_wave_sync(int site) { emu_wave_op(nullptr, 0, site, nullptr); }

template <class T>
static inline T emu_readlane(T v, int l, int site) {
  static_assert(sizeof(T) <= 64, "");
  const unsigned char* s = emu_wave_op(&v, sizeof(T), site, nullptr);
  T r;
  memcpy(&r, s + 64 * (l & 63), sizeof(T));
  return r;
}

static inline uint64_t emu_ballot(int p, int site) {
  const int b = p != 0;
  uint64_t m;
  const unsigned char* s = emu_wave_op(&b, sizeof(int), site, &m);
  uint64_t r = 0;
  for (int l = 0; l < 64; ++l)
    if (((m >> l) & 1) && *(const int*)(s + 64 * l)) r |= uint64_t(1) << l;
  return r;
}

template <class T>
static inline T emu_shfl_xor_(int site, T v, int mask, int width = 64) {
  const unsigned char* s = emu_wave_op(&v, sizeof(T), site, nullptr);
  const int self = emu_cur->lane;
  int idx = self ^ mask;
  if (idx >= ((self + width) & ~(width - 1))) idx = self;
  T r;
  memcpy(&r, s + 64 * idx, sizeof(T));
  return r;
}

// v_mfma_f32_4x4x1_16b_f32: 16 blocks of 4 lanes; in block b (lanes 4b..4b+3) lane 4b+j,
// register i accumulates A[i] B[j] with A[i] the a operand of lane 4b+i and B[j] the b of lane 4b+j
static inline emu_f4 emu_mfma_4x4x1(float a, float b, emu_f4 c, int site) {
  const float in[2] = {a, b};
  const unsigned char* s = emu_wave_op(in, sizeof(in), site, nullptr);
  const int L = emu_cur->lane, blk = L >> 2, j = L & 3;
  const float B = ((const float*)(s + 64 * (4 * blk + j)))[1];
  for (int i = 0; i < 4; ++i) c[i] = fmaf(((const float*)(s + 64 * (4 * blk + i)))[0], B, c[i]);
  return c;
}

// v_mfma_f32_16x16x4_f32: A[i][k] in lane i + 16k, B[k][j] in lane j + 16k, D[4g + r][j] in
// register r of lane j + 16g
static inline emu_f4 emu_mfma_16x16x4(float a, float b, emu_f4 c, int site) {
  const float in[2] = {a, b};
  const unsigned char* s = emu_wave_op(in, sizeof(in), site, nullptr);
  const int L = emu_cur->lane, j = L & 15, g = L >> 4;
  for (int r = 0; r < 4; ++r) {
    const int i = 4 * g + r;
    float acc = c[r];
    for (int k = 0; k < 4; ++k)
      acc = fmaf(((const float*)(s + 64 * (i + 16 * k)))[0], ((const float*)(s + 64 * (j + 16 * k)))[1], acc);
    c[r] = acc;
  }
  return c;
}

// v_mfma_f32_16x16x32_bf16: lane l holds eight k values of A row l & 15 and of B column l & 15
// (slot group l >> 4); D as for the fp32 instruction
static inline emu_f4 emu_mfma_16x16x32_bf16(emu_b8 a, emu_b8 b, emu_f4 c, int site) {
  struct { emu_b8 a, b; } in{a, b};
  const unsigned char* s = emu_wave_op(&in, sizeof(in), site, nullptr);
  const int L = emu_cur->lane, j = L & 15, g = L >> 4;
  for (int r = 0; r < 4; ++r) {
    const int i = 4 * g + r;
    float acc = c[r];
    for (int q = 0; q < 4; ++q) {
      emu_b8 av, bv;
      memcpy(&av, s + 64 * (i + 16 * q), sizeof(emu_b8));
      memcpy(&bv, s + 64 * (j + 16 * q) + sizeof(emu_b8), sizeof(emu_b8));
      for (int v = 0; v < 8; ++v) acc = fmaf((float)av[v], (float)bv[v], acc);
    }
    c[r] = acc;
  }
  return c;
}

template <class... A, size_t... I>
static inline void emu_invoke(void (*k)(A...), std::tuple<std::decay_t<A>...>& t, std::index_sequence<I...>) {
  k(std::get<I>(t)...);
}

extern "C" char __start_emu_lds[] __attribute__((weak, visibility("hidden")));
extern "C" char __stop_emu_lds[] __attribute__((weak, visibility("hidden")));

template <class... A>
static inline void emu_launch(const char* name, void (*k)(A...), EmuDim g, EmuDim b, void** params) {
  std::tuple<std::decay_t<A>...> t;
  size_t i = 0;
  std::apply([&](auto&... a) { ((memcpy((void*)&a, params[i++], sizeof(a))), ...); }, t);
  struct Ctx {
    void (*k)(A...);
    std::tuple<std::decay_t<A>...>* t;
  } ctx{k, &t};
  emu_set_lds(__start_emu_lds, __stop_emu_lds);
  emu_run_grid(name, g, b,
               [](void* c) {
                 auto* x = (Ctx*)c;
                 emu_invoke(x->k, *x->t, std::index_sequence_for<A...>{});
               },
               &ctx);
}
