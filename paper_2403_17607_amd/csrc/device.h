// Device-side helpers shared by the fused kernels.
#pragma once

#include <type_traits>

#include "common.h"

namespace ffmlp {

// Compile-time loop: f(std::integral_constant<int, I>) for I = B .. E-1.  Used
// where register arrays are indexed by the loop variable, so the index is a
// constant even when the body is too large for the unroller's heuristics.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// Two fp32 values to packed bf16 (low half = a), round-to-nearest-even
// (gfx950 v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  bf16x2 r = __builtin_convertvector(f32x2{a, b}, bf16x2);
  return __builtin_bit_cast(uint32_t, r);
}

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

// out += A * B on the matrix cores: 16x16 fp32 result, 32 bf16 contraction
// positions per lane group (see common.h for the lane layout).
__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(
      __builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ float act_apply(int act, float c) {
  switch (act) {
    case ACT_RELU: return c > 0.f ? c : 0.f;
    case ACT_SIGMOID: return 1.f / (1.f + __expf(-c));
    case ACT_SINE: return __sinf(c);
    default: return c;
  }
}

// Derivative of the output activation, from the pre-activation c and the
// fp32 output y = act(c) (both still in registers at the output layer).
__device__ __forceinline__ float act_out_grad(int act, float c, float y) {
  switch (act) {
    case ACT_RELU: return c > 0.f ? 1.f : 0.f;
    case ACT_SIGMOID: return y * (1.f - y);
    case ACT_SINE: return __cosf(c);
    default: return 1.f;
  }
}

// Derivative of a hidden activation from what the forward pass stored: the
// bf16 activation a (ReLU: a > 0, sigmoid: a (1 - a)) or, for sine, the
// stored bf16 cos(c) passed in as a.
template <int ACT>
__device__ __forceinline__ float act_hidden_grad(float a) {
  if constexpr (ACT == ACT_RELU) return a > 0.f ? 1.f : 0.f;
  else if constexpr (ACT == ACT_SIGMOID) return a * (1.f - a);
  else if constexpr (ACT == ACT_SINE) return a;
  else return 1.f;
}

template <int ACT>
__device__ __forceinline__ float act_hidden(float c) {
  if constexpr (ACT == ACT_RELU) return c > 0.f ? c : 0.f;
  else if constexpr (ACT == ACT_SIGMOID) return 1.f / (1.f + __expf(-c));
  else if constexpr (ACT == ACT_SINE) return __sinf(c);
  else return c;
}

// Cooperative copy of nfrag 1 KiB fragments from global memory into LDS.
__device__ __forceinline__ void copy_frags(u32x4* dst, const u32x4* src,
                                           uint32_t nfrag, int tid, int nthreads) {
  const uint32_t n = nfrag * 64u;
  for (uint32_t i = tid; i < n; i += nthreads) dst[i] = src[i];
}

// Deterministic wave-wide sum (fixed butterfly order).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace ffmlp
