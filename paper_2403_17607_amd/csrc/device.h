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

// Keep the computation of v at this point of the program: an empty asm
// that claims to change v, so the compiler can neither sink the work that
// produced v towards v's later uses nor drop it.  A layer's activations
// are otherwise converted only at the end of the layer, which keeps every
// strip's fp32 accumulators alive until then.
__device__ __forceinline__ void pin(uint32_t& v) { asm volatile("" : "+v"(v)); }

// ReLU of two packed bf16 values: a bf16 value is <= 0 exactly when its bit
// pattern read as int16 is <= 0, so a packed int16 max with 0 is ReLU.  It
// commutes with rounding (rounding keeps the sign), so ReLU may be applied
// after the conversion.
typedef short s16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t relu_bf16x2(uint32_t p) {
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(s16x2, p), (s16x2){0, 0}));
}

// Each half of p (a non-negative bf16 value) as 0 or 1 in that half.  The
// constant 1 in both halves comes from a register: an inline constant of a
// packed instruction would give the high half 0.
__device__ __forceinline__ uint32_t nonzero_halves(uint32_t p) {
  uint32_t m;
  asm("v_pk_min_u16 %0, %1, %2" : "=v"(m) : "v"(p), "v"(0x00010001u));
  return m;
}

// p with each 16-bit half multiplied by the 0 or 1 in the same half of m.
__device__ __forceinline__ uint32_t mask_halves(uint32_t p, uint32_t m) {
  uint32_t r;
  asm("v_pk_mul_lo_u16 %0, %1, %2" : "=v"(r) : "v"(p), "v"(m));
  return r;
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

// The training epilogue of one 16-row block of an output strip, OA the
// output activation: acc holds the pre-activations C (lane (g, i): row i,
// columns j0 .. j0 + 3), t the targets, `valid` which of the four are real
// (row < M, column < out_dim).  Returns Y as two packed bf16 pairs in y and
// the output delta scale (Y - T) sigma_out'(C) in d (0 where not valid), and
// adds (Y - T)^2 of the valid ones to loss.  Y and the loss use the fp32 Y.
template <int OA>
__device__ __forceinline__ void train_epilogue(const f32x4& acc, const u32x4& t, const bool (&valid)[4],
                                               float scale, float& loss, u32x2& y, u32x2& d) {
  float yv[4], dv[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    yv[q] = act_apply(OA, acc[q]);
    const float diff = yv[q] - __uint_as_float(t[q]);
    if (valid[q]) loss += diff * diff;
    dv[q] = valid[q] ? (scale * diff) * act_out_grad(OA, acc[q], yv[q]) : 0.f;
  }
  y = u32x2{pack_bf16x2(yv[0], yv[1]), pack_bf16x2(yv[2], yv[3])};
  d = u32x2{pack_bf16x2(dv[0], dv[1]), pack_bf16x2(dv[2], dv[3])};
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

// Buffer descriptor over [base, base + bytes) (gfx9 raw buffer, no
// swizzle).  The hardware range check makes loads past the end return 0 and
// drops stores past the end, so a wave can address its whole tile with
// 32-bit offsets and no per-row branches.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t kOOB = 0x80000000u;  // an offset past any descriptor's end

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const int n = bytes <= 0 ? 0 : (bytes > 0x7fffffff ? 0x7fffffff : (int)bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}
__device__ __forceinline__ u32x2 bload64(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
}
__device__ __forceinline__ u32x4 bload128(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ __forceinline__ uint32_t bload32(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0);
}
__device__ __forceinline__ uint32_t bload16(rsrc_t r, uint32_t voff, uint32_t soff) {
  return (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0);
}
// Stores are non-temporal (cache policy nt) by default: everything the
// forward and backward kernels store (outputs, the activation and delta
// stash, masks, dX) is read at most once, by a later kernel, so keeping it
// in L2 and the last-level cache would only evict lines that are still in
// use.  Measured on the training step: 4.7% faster at width 128 and 9% at
// width 64 (2^20 rows).  NT = false gives the default policy, whose stores
// are acknowledged sooner: a kernel that waits for all its stores at every
// layer (streamed weights) and gains nothing later uses it for inference.
constexpr int kStoreNT = 2;  // the nt bit of the buffer instructions' cache policy
template <bool NT = true>
__device__ __forceinline__ void bstore32(uint32_t v, rsrc_t r, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_buffer_store_b32(v, r, voff, soff, NT ? kStoreNT : 0);
}
template <bool NT = true>
__device__ __forceinline__ void bstore16(uint32_t v, rsrc_t r, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_buffer_store_b16((unsigned short)v, r, voff, soff, NT ? kStoreNT : 0);
}
template <bool NT = true>
__device__ __forceinline__ void bstore64(u32x2 v, rsrc_t r, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_buffer_store_b64(v, r, voff, soff, NT ? kStoreNT : 0);
}
template <bool NT = true>
__device__ __forceinline__ void bstore128(u32x4 v, rsrc_t r, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, voff, soff, NT ? kStoreNT : 0);
}

// Asynchronous copy of nfrag 1 KiB fragments from global memory into LDS
// with direct-to-LDS loads (no registers): wave w copies fragments w,
// w + nwaves, ...; lane l of a load writes bytes 16 l .. 16 l + 15 of the
// fragment.  The data is in LDS once the issuing wave has waited for its
// vector memory counter; other waves may read it after a barrier.
__device__ __forceinline__ void stage_frags(u32x4* dst, const u32x4* src, uint32_t nfrag,
                                            int wave, int nwaves, int lane) {
  for (uint32_t f = wave; f < nfrag; f += nwaves)
    __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)(src + (size_t)f * 64 + lane),
                                     (void __attribute__((address_space(3)))*)(dst + (size_t)f * 64), 16, 0, 0);
}

// Wait for every vector memory operation of this wave (direct-to-LDS loads
// included), then synchronize the workgroup.
__device__ __forceinline__ void drain_and_sync() {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
}

// Deterministic wave-wide sum (fixed butterfly order).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace ffmlp
