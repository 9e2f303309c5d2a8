// Weight gradients G_i = A_i^T D_{i+1} of Algorithm 2 (arXiv 2403.17607,
// section III-A), a contraction over the whole batch, plus the fixed-order
// reduction of the per-workgroup partial sums and the weight packing.
//
// The paper computes these products outside its fused kernel with library
// GEMMs; here one kernel covers every layer (grid.y = layer) as a split-K
// MFMA contraction: workgroup p of a layer sums its own contiguous range of
// batch rows into an fp32 partial G, and a second kernel adds the P partials
// in a fixed order, so G is bitwise reproducible.
//
// A matrix-core operand for a contraction over the batch needs eight batch
// rows of one feature per lane, while the stash holds each batch row's
// features together.  Each chunk of rows is therefore transposed on its way
// into LDS (feature-major, batch contiguous), and every operand fragment is
// then a single 16-byte LDS read.
#include "device.h"

namespace ffmlp {

template <int W>
__global__ __launch_bounds__(256) void wgrad_kernel(const WgradArgs a) {
  using C = WgCfg<W>;
  constexpr int TBK = C::TBK, TBJ = C::TBJ, GJ = C::GJ, KS = C::KS, KSW = C::KSW;
  constexpr int CH = wg_chunk<W>();
  constexpr int LDT = CH + 8;  // LDS row stride (elements) of the transposed tiles
  extern __shared__ u32x4 smem_v[];
  uint16_t* AT = reinterpret_cast<uint16_t*>(smem_v);
  uint16_t* DT = AT + W * LDT;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int li = lane & 15, lg = lane >> 4;
  const int l = blockIdx.y, p = blockIdx.x, L = a.L;
  const int64_t M = a.M;
  const int fan_in = (l == 0) ? a.in_dim : W;
  const int fan_out = (l == L - 1) ? a.out_dim : W;
  const int OP = ((a.out_dim + 15) >> 4) * 16;
  const int KT = (fan_in + 15) >> 4, JT = (fan_out + 15) >> 4;
  const int wks = wave % KS, rest = wave / KS;
  const int wj = rest % GJ, wk = rest / GJ;

  const uint16_t* dsrc = (l == L - 1) ? a.deltaOut : a.deltaH + (size_t)l * a.M16 * W;
  const int dF = (l == L - 1) ? OP : W;
  const uint16_t* asrc = (l == 0) ? nullptr : a.stashA + (size_t)(l - 1) * a.M16 * W;
  const bool xvec = (a.in_dim & 7) == 0;

  f32x4 acc[TBK][TBJ];
#pragma unroll
  for (int i = 0; i < TBK; ++i)
#pragma unroll
    for (int j = 0; j < TBJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int64_t nch = (M + CH - 1) / CH;
  const int64_t c_begin = (int64_t)p * a.chunks_per_block;
  int64_t c_end = c_begin + a.chunks_per_block;
  if (c_end > nch) c_end = nch;

  for (int64_t c = c_begin; c < c_end; ++c) {
    const int64_t c0 = c * CH;
    __syncthreads();
    // ---- A chunk -> AT[f][m] ----
    if (l == 0) {
      const int in_dim = a.in_dim;
      if (xvec) {
        const int units = CH * in_dim / 8;
        for (int u = tid; u < units; u += 256) {
          const int e = u * 8;
          const int ml = e / in_dim, f = e - ml * in_dim;
          const int64_t row = c0 + ml;
          u32x4 v = {0u, 0u, 0u, 0u};
          if (row < M) v = *reinterpret_cast<const u32x4*>(a.X + row * in_dim + f);
          uint16_t* t = AT + (size_t)f * LDT + ml;
          t[0 * LDT] = (uint16_t)(v.x & 0xffff);
          t[1 * LDT] = (uint16_t)(v.x >> 16);
          t[2 * LDT] = (uint16_t)(v.y & 0xffff);
          t[3 * LDT] = (uint16_t)(v.y >> 16);
          t[4 * LDT] = (uint16_t)(v.z & 0xffff);
          t[5 * LDT] = (uint16_t)(v.z >> 16);
          t[6 * LDT] = (uint16_t)(v.w & 0xffff);
          t[7 * LDT] = (uint16_t)(v.w >> 16);
        }
      } else {
        const int units = CH * in_dim;
        for (int u = tid; u < units; u += 256) {
          const int ml = u / in_dim, f = u - ml * in_dim;
          const int64_t row = c0 + ml;
          AT[(size_t)f * LDT + ml] = (row < M) ? a.X[row * in_dim + f] : (uint16_t)0;
        }
      }
    }
    // Tile-image sources: 8 elements = rows i, i+1 (i even) x features
    // 16 s + 4 g + 0..3 of one 16-row block.
    for (int pass = (l == 0) ? 1 : 0; pass < 2; ++pass) {
      const uint16_t* src = pass == 0 ? asrc : dsrc;
      const int F = pass == 0 ? W : dF;
      uint16_t* T = pass == 0 ? AT : DT;
      const int units = CH * F / 8;
      for (int u = tid; u < units; u += 256) {
        const int e = u * 8;
        const int tl = e / (16 * F);
        const int rem = e - tl * 16 * F;
        const int s = rem >> 8, w = rem & 255;
        const int ln = w >> 2, g = ln >> 4, i = ln & 15;
        const int64_t row = c0 + 16 * tl + i;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (c0 + 16 * tl < M) v = *reinterpret_cast<const u32x4*>(src + (size_t)c0 * F + e);
        if (row >= M) { v.x = 0u; v.y = 0u; }
        if (row + 1 >= M) { v.z = 0u; v.w = 0u; }
        const int f = 16 * s + 4 * g;
        uint32_t* t = reinterpret_cast<uint32_t*>(T + (size_t)f * LDT + 16 * tl + i);
        constexpr int LDW = LDT / 2;
        t[0 * LDW] = (v.x & 0xffffu) | (v.z << 16);
        t[1 * LDW] = (v.x >> 16) | (v.z & 0xffff0000u);
        t[2 * LDW] = (v.y & 0xffffu) | (v.w << 16);
        t[3 * LDW] = (v.y >> 16) | (v.w & 0xffff0000u);
      }
    }
    __syncthreads();
    // ---- contraction over the chunk's batch rows ----
#pragma unroll
    for (int q = 0; q < KSW; ++q) {
      const int koff = (wks * KSW + q) * 32 + lg * 8;
      u32x4 af[TBK], bfr[TBJ];
#pragma unroll
      for (int tk = 0; tk < TBK; ++tk) {
        const int kt = wk * TBK + tk;
        af[tk] = (kt < KT) ? *reinterpret_cast<const u32x4*>(AT + (size_t)(16 * kt + li) * LDT + koff)
                           : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int tj = 0; tj < TBJ; ++tj) {
        const int jt = wj * TBJ + tj;
        bfr[tj] = (jt < JT) ? *reinterpret_cast<const u32x4*>(DT + (size_t)(16 * jt + li) * LDT + koff)
                            : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int tk = 0; tk < TBK; ++tk)
#pragma unroll
        for (int tj = 0; tj < TBJ; ++tj)
          if (wk * TBK + tk < KT && wj * TBJ + tj < JT) acc[tk][tj] = mfma16(af[tk], bfr[tj], acc[tk][tj]);
    }
  }

  // Waves that split the batch add up in a fixed order.
  if constexpr (KS > 1) {
    __syncthreads();
    f32x4* red = reinterpret_cast<f32x4*>(smem_v);
    const int blk = wave / KS;
    if (wks != 0) {
#pragma unroll
      for (int tk = 0; tk < TBK; ++tk)
#pragma unroll
        for (int tj = 0; tj < TBJ; ++tj)
          red[(((blk * (KS - 1) + wks - 1) * TBK + tk) * TBJ + tj) * 64 + lane] = acc[tk][tj];
    }
    __syncthreads();
    if (wks != 0) return;
#pragma unroll
    for (int k = 1; k < KS; ++k)
#pragma unroll
      for (int tk = 0; tk < TBK; ++tk)
#pragma unroll
        for (int tj = 0; tj < TBJ; ++tj)
          acc[tk][tj] += red[(((blk * (KS - 1) + k - 1) * TBK + tk) * TBJ + tj) * 64 + lane];
  }

  // Partial G of this workgroup, in the weights' own layout.
  int64_t off = 0;
  if (l >= 1) off = (int64_t)a.in_dim * W + (int64_t)(l - 1) * W * W;
  float* dst = a.partial + (int64_t)p * a.params + off;
#pragma unroll
  for (int tk = 0; tk < TBK; ++tk) {
#pragma unroll
    for (int tj = 0; tj < TBJ; ++tj) {
      const int kt = wk * TBK + tk, jt = wj * TBJ + tj;
      if (kt >= KT || jt >= JT) continue;
      const int j = 16 * jt + li;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int k = 16 * kt + 4 * lg + r;
        if (k < fan_in && j < fan_out) dst[(int64_t)k * fan_out + j] = acc[tk][tj][r];
      }
    }
  }
}

__global__ __launch_bounds__(256) void reduce_kernel(const ReduceArgs a) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e < a.params) {
    float s = 0.f;
    for (int p = 0; p < a.P; ++p) s += a.partial[(int64_t)p * a.params + e];
    a.G[e] = s;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0 && a.loss != nullptr) {
    float s = 0.f;
    for (int i = 0; i < a.nloss; ++i) s += a.lossPart[i];
    *a.loss = s * a.loss_scale;
  }
}

// One thread per packed bf16 element: fragment (strip, k-block), lane,
// slot; see common.h for the two orientations and the contraction orders.
__global__ __launch_bounds__(256) void pack_kernel(const PackArgs a) {
  const int64_t n = (int64_t)a.strips * a.kblocks * 512;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= n) return;
  const int slot = (int)(e & 7), lane = (int)((e >> 3) & 63);
  const int frag = (int)(e >> 9);
  const int s = frag / a.kblocks, kb = frag - s * a.kblocks;
  const int g = lane >> 4, row = 16 * s + (lane & 15);
  int pos;  // contraction index the (g, slot) pair stands for
  if (a.first)
    pos = 32 * kb + 8 * g + slot;
  else
    pos = 32 * kb + (slot < 4 ? 4 * g + slot : 16 + 4 * g + (slot - 4));
  int f, j;  // W[f][j]
  if (a.dir == 0) { f = pos; j = row; } else { f = row; j = pos; }
  uint16_t v = 0;
  if (f < a.fan_in && j < a.fan_out) v = a.W[(int64_t)f * a.fan_out + j];
  a.dst[e] = v;
}

template <int W>
static hipError_t wgrad_t(const WgradArgs& a, hipStream_t stream) {
  using C = WgCfg<W>;
  constexpr int CH = wg_chunk<W>();
  size_t lds = (size_t)2 * W * (CH + 8) * 2;
  if constexpr (C::KS > 1) {
    const size_t red = (size_t)C::GK * C::GJ * (C::KS - 1) * C::TBK * C::TBJ * 64 * 16;
    if (red > lds) lds = red;
  }
  auto kern = wgrad_kernel<W>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(a.P, a.L), dim3(256), lds, stream, a);
  return hipGetLastError();
}

hipError_t launch_wgrad(int width, const WgradArgs& a, hipStream_t s) {
  switch (width) {
    case 16: return wgrad_t<16>(a, s);
    case 32: return wgrad_t<32>(a, s);
    case 64: return wgrad_t<64>(a, s);
    case 128: return wgrad_t<128>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_reduce(const ReduceArgs& a, hipStream_t s) {
  int64_t blocks = (a.params + 255) / 256;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_pack(const PackArgs& a, hipStream_t s) {
  const int64_t n = (int64_t)a.strips * a.kblocks * 512;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(pack_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace ffmlp
