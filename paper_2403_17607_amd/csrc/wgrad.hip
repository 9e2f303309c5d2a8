// Weight gradients G_i = A_i^T D_{i+1} of Algorithm 2 (arXiv 2403.17607,
// section III-A), a contraction over the whole batch, plus the fixed-order
// reduction of the per-workgroup partial sums and the weight packing.
//
// The paper computes these products outside its fused kernel with library
// GEMMs; here one kernel covers every layer (grid.y = layer) as a split-K
// MFMA contraction: workgroup p of a layer sums its own contiguous range of
// batch rows into an fp32 partial G, and two small passes add the P partials
// in a fixed order, so G is bitwise reproducible.
//
// A matrix-core operand for a contraction over the batch needs eight batch
// rows of one feature per lane, while the stash holds each batch row's
// features together.  Each chunk of rows is therefore transposed on its way
// into LDS (feature-major, batch contiguous), and every operand fragment is
// then a single 16-byte LDS read.  The next chunk's global loads are issued
// into registers before the current chunk's MFMAs, so HBM traffic overlaps
// the contraction.
#include "device.h"

namespace ffmlp {

template <int W>
__global__ __launch_bounds__(256) void wgrad_kernel(const WgradArgs a) {
  using C = WgCfg<W>;
  constexpr int TBK = C::TBK, TBJ = C::TBJ, GJ = C::GJ, KS = C::KS, KSW = C::KSW;
  constexpr int CH = wg_chunk<W>();
  // Chunk loads are non-temporal at widths up to 32: every byte is read
  // once (training step at 2^20 rows: width 16 188 -> 165 us, width 32
  // 290 -> 265 us); at width 128 the same policy measured 2-5% slower.
  constexpr int kLoadPol = W <= 32 ? 2 : 0;
  constexpr int LDT = CH + 8;      // LDS row stride (bf16) of the transposed tiles
  constexpr int LDW = LDT / 2;     // the same in 32-bit words
  constexpr int UPT = CH * W / 8 / 256;  // 16-byte units per thread per tensor
  static_assert(UPT >= 2 && UPT % 2 == 0, "chunk geometry");
  extern __shared__ u32x4 smem_v[];
  uint16_t* AT = reinterpret_cast<uint16_t*>(smem_v);
  uint16_t* DT = AT + W * LDT;
  uint32_t* AT32 = reinterpret_cast<uint32_t*>(AT);
  uint32_t* DT32 = reinterpret_cast<uint32_t*>(DT);

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int li = lane & 15, lg = lane >> 4;
  const int l = blockIdx.y, p = blockIdx.x, L = a.L;
  const int64_t M = a.M;
  const int in_dim = a.in_dim;
  const int fan_in = (l == 0) ? in_dim : W;
  const int fan_out = (l == L - 1) ? a.out_dim : W;
  const int OP = ((a.out_dim + 15) >> 4) * 16;
  const int KT = (fan_in + 15) >> 4, JT = (fan_out + 15) >> 4;
  const int wks = wave % KS, rest = wave / KS;
  const int wj = rest % GJ, wk = rest / GJ;

  const uint16_t* dsrc = (l == L - 1) ? a.deltaOut : a.deltaH + (size_t)l * a.M16 * W;
  const int dF = (l == L - 1) ? OP : W;
  const uint16_t* asrc = (l == 0) ? a.X : a.stashA + (size_t)(l - 1) * a.M16 * W;
  const bool xvec = (in_dim & 7) == 0;
  const int nf8 = (in_dim + 7) >> 3;  // 8-feature groups of an X row

  u32x4 ra[UPT], rd[UPT];

  // ---- global -> registers: buffer loads ----
  // A chunk of a tensor is read through a buffer descriptor whose base is
  // the chunk's first byte and whose size is the chunk's valid bytes; the
  // hardware returns zeros past that size, which covers rows past the
  // batch.  (Stash rows between M and the next multiple of 16 hold finite
  // activations and exactly zero deltas, so they add nothing to G.)  The
  // per-unit byte offsets do not depend on the chunk and are computed once.
  //
  // Tile-image tensor with F features: unit v covers rows 16 tl + 2 ip,
  // +1 and features 16 s + 4 g + 0..3, and sits at byte 16 v of the chunk,
  // so a wave reads 1 KiB in one piece.  The transposed LDS writes of each
  // half-wave (ip and g vary) still hit 32 distinct banks.
  struct TileUnit {
    int tl, s, g, ip;
  };
  auto tile_unit = [&](int v, int S) {
    const int ip = v & 7, g = (v >> 3) & 3, rest = v >> 5;
    return TileUnit{rest / S, rest % S, g, ip};
  };
  // Byte offset of unit v inside the chunk (past the chunk when v >= U).
  auto tile_voff = [&](int v) { return (uint32_t)(v * 16); };
  const bool xmode = (l == 0);
  uint32_t voa[UPT], vod[UPT];
  {
#pragma unroll
    for (int k = 0; k < UPT; ++k) {
      vod[k] = tile_voff(k * 256 + tid);  // >= the chunk size when past it
      voa[k] = vod[k];
    }
    if (xmode) {
      // X (row-major, in_dim a multiple of 8): unit pair q covers rows
      // 2 j, 2 j + 1 and features 8 f8 .. + 7; consecutive lanes take
      // consecutive j.
      const int npairs = (CH / 2) * nf8;
#pragma unroll
      for (int k = 0; k < UPT / 2; ++k) {
        const int q = k * 256 + tid;
        const int j = q % (CH / 2), f0 = (q / (CH / 2)) * 8;
        const uint32_t past = (uint32_t)(CH * in_dim * 2);
        voa[2 * k] = q < npairs ? (uint32_t)((2 * j * in_dim + f0) * 2) : past;
        voa[2 * k + 1] = q < npairs ? (uint32_t)(((2 * j + 1) * in_dim + f0) * 2) : past;
      }
    }
  }
  auto rsrc = [&](const uint16_t* base, int64_t c0, int row_bytes, int64_t rows_valid) {
    int64_t rows = rows_valid - c0;
    if (rows > CH) rows = CH;
    if (rows < 0) rows = 0;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base) + c0 * (row_bytes / 2),
                                             (short)0, (int)(rows * row_bytes), 0x00020000);
  };
  auto load_chunk = [&](int64_t c) {
    const int64_t c0 = c * CH;
    const __amdgpu_buffer_rsrc_t rd_src = rsrc(dsrc, c0, dF * 2, a.M16);
    const __amdgpu_buffer_rsrc_t ra_src =
        xmode ? rsrc(a.X, c0, in_dim * 2, xvec ? M : 0) : rsrc(asrc, c0, W * 2, a.M16);
#pragma unroll
    for (int k = 0; k < UPT; ++k) ra[k] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(ra_src, voa[k], 0, kLoadPol));
#pragma unroll
    for (int k = 0; k < UPT; ++k) rd[k] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rd_src, vod[k], 0, kLoadPol));
  };

  // ---- registers -> LDS, transposed to [feature][batch row] ----
  auto store_tile = [&](const u32x4 (&r)[UPT], uint32_t* T32, int F) {
    const int S = F >> 4;
    const int U = CH * F / 8;
#pragma unroll
    for (int k = 0; k < UPT; ++k) {
      const int v = k * 256 + tid;
      if (v < U) {
        const TileUnit t = tile_unit(v, S);
        const u32x4 x = r[k];
        uint32_t* d = T32 + (16 * t.s + 4 * t.g) * LDW + 8 * t.tl + t.ip;
        d[0 * LDW] = (x.x & 0xffffu) | (x.z << 16);
        d[1 * LDW] = (x.x >> 16) | (x.z & 0xffff0000u);
        d[2 * LDW] = (x.y & 0xffffu) | (x.w << 16);
        d[3 * LDW] = (x.y >> 16) | (x.w & 0xffff0000u);
      }
    }
  };
  auto store_x = [&](const u32x4 (&r)[UPT]) {
    const int npairs = (CH / 2) * nf8;
#pragma unroll
    for (int k = 0; k < UPT / 2; ++k) {
      const int q = k * 256 + tid;
      if (q < npairs) {
        const int j = q % (CH / 2), f0 = (q / (CH / 2)) * 8;
        const u32x4 x0 = r[2 * k], x1 = r[2 * k + 1];
        const uint32_t w0[4] = {x0.x, x0.y, x0.z, x0.w}, w1[4] = {x1.x, x1.y, x1.z, x1.w};
        uint32_t* d = AT32 + f0 * LDW + j;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          d[(2 * e) * LDW] = (w0[e] & 0xffffu) | (w1[e] << 16);
          d[(2 * e + 1) * LDW] = (w0[e] >> 16) | (w1[e] & 0xffff0000u);
        }
      }
    }
  };
  // Other input widths: X goes straight from global memory into LDS,
  // element by element, when the chunk is stored (no register staging).
  auto copy_x_scalar = [&](int64_t c0) {
    for (int u = tid; u < CH * in_dim; u += 256) {
      const int ml = u / in_dim, f = u - ml * in_dim;
      const int64_t row = c0 + ml;
      AT[(size_t)f * LDT + ml] = row < M ? a.X[row * in_dim + f] : (uint16_t)0;
    }
  };

  f32x4 acc[TBK][TBJ];
#pragma unroll
  for (int i = 0; i < TBK; ++i)
#pragma unroll
    for (int j = 0; j < TBJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int64_t nch = (M + CH - 1) / CH;
  const int64_t c_begin = (int64_t)p * a.chunks_per_block;
  int64_t c_end = c_begin + a.chunks_per_block;
  if (c_end > nch) c_end = nch;

  if (c_begin < c_end) load_chunk(c_begin);
  for (int64_t c = c_begin; c < c_end; ++c) {
    __syncthreads();  // every wave is done reading the previous chunk
    if (!xmode) store_tile(ra, AT32, W);
    else if (xvec) store_x(ra);
    else copy_x_scalar(c * CH);
    store_tile(rd, DT32, dF);
    __syncthreads();
    if (c + 1 < c_end) load_chunk(c + 1);
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
    for (int k = 1; k < KS; ++k) {
#pragma unroll
      for (int tk = 0; tk < TBK; ++tk)
#pragma unroll
        for (int tj = 0; tj < TBJ; ++tj)
          acc[tk][tj] += red[(((blk * (KS - 1) + k - 1) * TBK + tk) * TBJ + tj) * 64 + lane];
      __builtin_amdgcn_sched_barrier(0);  // one partial at a time: bounds the registers
    }
  }

  // Partial G of this workgroup, in the weights' own layout.
  int64_t off = 0;
  if (l >= 1) off = (int64_t)in_dim * W + (int64_t)(l - 1) * W * W;
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

// Fixed-order sum of the P partials into G, one pass.  Block b owns
// parameters 64 b .. 64 b + 63 and its wave y (of 16) adds slice y of the
// partials, [y P / 16, (y + 1) P / 16), in order; the 16 slice sums are then
// added in order through LDS.  The last block instead sums the loss
// partials: thread t < 256 adds partials t, t + 256, ... in order, then a
// fixed tree over those 256 threads.
static_assert(kReduceSlices * 64 == 1024, "one wave per slice in a 1024-thread block");
__global__ __launch_bounds__(1024) void reduce_kernel(const ReduceArgs a) {
  __shared__ float part[kReduceSlices][64];
  const int t = threadIdx.x;
  if (blockIdx.x == gridDim.x - 1) {
    float* lp = &part[0][0];  // 256 of its 1024 floats
    if (t < 256) {
      float s = 0.f;
      for (int i = t; i < a.nloss; i += 256) s += a.lossPart[i];
      lp[t] = s;
    }
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
      if (t < h) lp[t] += lp[t + h];
      __syncthreads();
    }
    if (t == 0 && a.loss != nullptr) *a.loss = lp[0] * a.loss_scale;
    return;
  }
  const int j = t & 63, y = t >> 6;
  const int64_t e = (int64_t)blockIdx.x * 64 + j;
  float s = 0.f;
  if (e < a.params) {
    const int p0 = (int)((int64_t)a.P * y / kReduceSlices);
    const int p1 = (int)((int64_t)a.P * (y + 1) / kReduceSlices);
    // Loads go out eight at a time, then are added in order: the same sum,
    // without one memory latency per partial.
    const float* src = a.partial + e;
    int p = p0;
    for (; p + 8 <= p1; p += 8) {
      float v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = src[(int64_t)(p + k) * a.params];
#pragma unroll
      for (int k = 0; k < 8; ++k) s += v[k];
    }
    for (; p < p1; ++p) s += src[(int64_t)p * a.params];
  }
  part[y][j] = s;
  __syncthreads();
  if (t < 64 && e < a.params) {
    float g = 0.f;
#pragma unroll
    for (int k = 0; k < kReduceSlices; ++k) g += part[k][t];
    a.G[e] = g;
  }
}

// One thread per packed bf16 element.  The buffer holds the forward
// layers 0 .. L-1, then the backward layers 1 .. L-1, then the backward
// layer 0 (for the input gradient), each as fragments
// [strip][k-block][lane][slot]; see common.h for the two orientations and
// the contraction orders.
__global__ __launch_bounds__(256) void pack_kernel(const PackArgs a) {
  const int64_t e0 = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e0 >= a.total) return;
  const int Wd = a.width, L = a.L;
  auto fan_in = [&](int l) { return l == 0 ? a.in_dim : Wd; };
  auto fan_out = [&](int l) { return l == L - 1 ? a.out_dim : Wd; };
  // Locate the layer and orientation of element e0: forward layers
  // 0 .. L-1, backward layers 1 .. L-1, then backward layer 0 (read only
  // by the input-gradient step).  A segment holds strips(rows) fragments of
  // 512 elements per k-block, rows being the fan_out (forward) or fan_in
  // (backward) of its layer, so every hidden segment has the same size and
  // the position follows in closed form, whatever the depth.
  const int64_t per = (int64_t)((Wd + 31) / 32) * 512;  // one strip
  const int64_t nW = per * ((Wd + 15) / 16);
  const int64_t nO = per * ((a.out_dim + 15) / 16);
  const int64_t nH = (int64_t)(L - 1) * nW;  // L - 1 segments of nW
  int64_t e = e0;
  int dir, l;
  if (e < nH) {
    dir = 0;
    l = (int)(e / nW);
    e -= (int64_t)l * nW;
  } else if ((e -= nH) < nO) {
    dir = 0;
    l = L - 1;
  } else if ((e -= nO) < nH) {
    dir = 1;
    l = 1 + (int)(e / nW);
    e -= (int64_t)(l - 1) * nW;
  } else {
    e -= nH;  // < strips(in_dim) strips: e0 < total
    dir = 1;
    l = 0;
  }
  const int64_t woff = l == 0 ? 0 : (int64_t)a.in_dim * Wd + (int64_t)(l - 1) * Wd * Wd;
  const int fi = fan_in(l), fo = fan_out(l);
  const int kblocks = (Wd + 31) / 32;  // every layer is padded to the width's k-blocks
  const int slot = (int)(e & 7), lane = (int)((e >> 3) & 63);
  const int frag = (int)(e >> 9);
  const int s = frag / kblocks, kb = frag - s * kblocks;
  const int g = lane >> 4, row = 16 * s + (lane & 15);
  int pos;  // contraction index the (g, slot) pair stands for
  if (dir == 0 && l == 0)
    pos = 32 * kb + 8 * g + slot;
  else
    pos = 32 * kb + (slot < 4 ? 4 * g + slot : 16 + 4 * g + (slot - 4));
  int f, j;  // W_l[f][j]
  if (dir == 0) { f = pos; j = row; } else { f = row; j = pos; }
  uint16_t v = 0;
  if (f < fi && j < fo) v = a.W[woff + (int64_t)f * fo + j];
  a.dst[e0] = v;
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
  int occ = 0;
  hipError_t e = kernel_occupancy(reinterpret_cast<const void*>(kern), 256, lds, &occ);
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
  const int64_t blocks = (a.params + 63) / 64;  // plus one for the loss
  hipLaunchKernelGGL(reduce_kernel, dim3((unsigned)blocks + 1), dim3(1024), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_pack(const PackArgs& a, hipStream_t s) {
  if (a.total == 0) return hipSuccess;
  hipLaunchKernelGGL(pack_kernel, dim3((unsigned)((a.total + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace ffmlp
