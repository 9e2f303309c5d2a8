// Fused forward kernel: inference (Algorithm 1) and the forward half of the
// training step (Algorithm 2: keep every activation, then the L2 loss and
// the output delta), arXiv 2403.17607 section III-A.
//
// One workgroup owns NW * NT * 16 batch rows at a time (persistent loop
// over row tiles).  Each wave keeps the activations of its NT 16-row blocks
// in VGPRs across all layers as MFMA B operands; a layer is the transposed
// product C^T = W^T A^T on the matrix cores, with the packed weights read
// from LDS as the A operand.  When every layer's packed weights fit in LDS
// they are loaded once per workgroup; otherwise each layer is staged in
// turn (section III-B stages one weight matrix at a time in shared local
// memory).  HBM is touched for X, Y and, when training, T and the stash.
//
// The weight fragments of the next strip are read from LDS while the
// current strip's MFMAs run (across the layer boundary too when all layers
// are resident).  Global memory is addressed through one buffer descriptor
// per wave tile, whose range check replaces per-row bounds branches.
#pragma once

#include "device.h"

namespace ffmlp {

// Weight fragments of strip s.  Every packed layer has KBW k-blocks (the
// first layer's are zero-padded past in_dim), so the count is a constant.
template <int KBW>
__device__ __forceinline__ void load_frags(const u32x4* wl, int s, int lane, u32x4 (&af)[KBW]) {
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb) af[kb] = wl[(s * KBW + kb) * 64 + lane];
}

// acc[n] = (one 16-feature strip of the packed layer) x act[n].
template <int NT, int KBW>
__device__ __forceinline__ void strip_product(const u32x4 (&af)[KBW], const u32x4 (&act)[NT][KBW],
                                              f32x4 (&acc)[NT]) {
#pragma unroll
  for (int n = 0; n < NT; ++n) acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb)
#pragma unroll
    for (int n = 0; n < NT; ++n) acc[n] = mfma16(af[kb], act[n][kb], acc[n]);
}

// RES: every layer's weights resident in LDS (else staged layer by layer).
// FU selects the tile loop: 0 general; 1 and 2 the fused last layers (see
// below) for L odd and L even.  Each combination is its own kernel, so that
// the register allocation of one loop does not constrain another and no
// loop carries the other's branches (whose joins force conservative waits
// on LDS loads).
// SMALL: one 16-row block per wave (batches that give the usual tiles
// fewer than two per compute unit, widths up to 64): four times as many
// workgroups, so more waves share each CU's latency.
// Waves per workgroup: inference at widths up to 32, and the small-batch
// variant at any width, stream X and Y with little arithmetic per byte and
// run 8 waves (more bytes in flight per CU: width 16 at 2^22 rows 66 -> 56
// us, width 64 at 2^17 rows 12.6 -> 11.0 us); every other case uses the
// tile configuration.  The row tile changes with it; the stash layout
// does not.
// Width-128 inference runs two 16-row blocks per wave and 16 waves per
// workgroup (4 per SIMD instead of 2 with four blocks and 8 waves: more
// waves to hide the latencies of the layer transitions and the X loads;
// the fragment reads per row double, a quarter of LDS bandwidth at the full
// MFMA rate).  Measured at 2^20 rows: 5 matrices 112.1 -> 106.5 us, depth 16
// with streamed weights 494.6 -> 474.1 us.  The even-L fused loop (FU 2)
// needs more registers than the 128 that 4 waves per SIMD leave and runs 12
// waves (97.7 -> 93.5 us for 4 matrices).
template <int W, int MODE, bool SMALL = false, int FU = 0>
constexpr int fwd_waves() {
  if constexpr (W == 128 && MODE == FWD_INFER && !SMALL) return FU == 2 ? 12 : 16;
  return (SMALL || (W <= 32 && MODE == FWD_INFER)) ? 8 : TileCfg<W>::NW;
}
// 16-row blocks per wave.
template <int W, int MODE, bool SMALL = false, int FU = 0>
constexpr int fwd_nt() {
  if constexpr (SMALL) return 1;
  if constexpr (W == 128 && MODE == FWD_INFER) return 2;
  return TileCfg<W>::NT;
}

// TST (training forward at width 128, for the fused backward): each
// 512-byte strip of a block in stashA holds the strip transposed, lane
// (g, n) feature 16 s + n of rows 4 g .. 4 g + 3, instead of lane (g, i)
// row i of features 16 s + 4 g .. + 3.  The fused backward reads it as the
// A operand of G_l directly; otherwise it transposes every strip on the
// matrix cores itself (8 MFMAs and their conversions per layer and wave,
// on its critical path), where the forward, bound by HBM, has them to
// spare.  Same bytes, same addresses.
template <int W, int ACT, int MODE, int FU, bool RES, bool SMALL = false, bool LIN = false, bool TST = false>
__global__ __launch_bounds__((fwd_waves<W, MODE, SMALL, FU>() * 64)) void fwd_kernel(const FwdArgs a) {
  constexpr int NT = fwd_nt<W, MODE, SMALL, FU>(), NW = fwd_waves<W, MODE, SMALL, FU>();
  constexpr int KBW = (W + 31) / 32, SW = W / 16;
  extern __shared__ u32x4 smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int li = lane & 15, lg = lane >> 4;
  const int L = a.L, in_dim = a.in_dim, out_dim = a.out_dim;
  const int64_t M = a.M;
  const int KB0 = (in_dim + 31) >> 5;
  const int SO = (out_dim + 15) >> 4;
  const int OP = SO * 16;
  const bool xvec = (in_dim & 7) == 0;
  const bool yvec = (out_dim & 3) == 0;
  const int out_act = LIN ? (int)ACT_LINEAR : a.out_act;
  static_assert(!TST || (MODE == FWD_TRAIN && NT % 2 == 0), "transposed stash: training forward, block pairs");
  // TST: 0/1 selection matrices; an MFMA of a block pair's strip (block n in
  // slots 0-3, block n + 1 in slots 4-7) against sel0 (sel1) gives block n
  // (n + 1) transposed, exactly.
  u32x4 sel0 = {0u, 0u, 0u, 0u}, sel1 = {0u, 0u, 0u, 0u};
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
  if constexpr (TST) {
    const int q = li - 4 * lg;
    if (q >= 0 && q < 4) {
      const uint32_t one = 0x3F80u << (16 * (q & 1));
      if (q < 2) {
        sel0.x = one;
        sel1.z = one;
      } else {
        sel0.y = one;
        sel1.w = one;
      }
    }
  }
  constexpr bool resident = RES;
  // Non-temporal stores, except for inference with streamed weights: there
  // every layer ends by waiting for all outstanding memory operations, the
  // output stores included, and nothing reads Y soon after.
  constexpr bool NTS = RES || MODE != FWD_INFER;
  const int G = gridDim.x;
  auto layer_off = [&](int l) -> uint32_t {
    return l == 0 ? 0u : a.lay0_frags + (uint32_t)(l - 1) * a.layH_frags;
  };

  // Weights: all layers resident in LDS, or (too large) layers staged in
  // turn through two LDS buffers: while layer l computes from one buffer,
  // the next layer (the first layer of the next tile after the last one)
  // is loaded into the other with direct-to-LDS loads.  One barrier per
  // layer.  `step` counts the layers this workgroup has run; its parity
  // picks the buffer.
  const uint32_t bufq = (uint32_t)((L > 1 ? SW : SO) * KBW) * 64;  // one buffer, in u32x4
  int step = 0;
  auto stream_buf = [&](int st) { return smem + ((st & 1) ? bufq : 0u); };
  auto stage_layer = [&](int l, int st) {
    const uint32_t nf = (uint32_t)((l == L - 1 ? SO : SW) * KBW);
    stage_frags(stream_buf(st), a.packed + (size_t)layer_off(l) * 64, nf, wave, NW, lane);
  };
  // Weight loads are issued here and waited for after the first X loads
  // below, so the two overlap.
  if (resident) {
    stage_frags(smem, a.packed, a.total_frags, wave, NW, lane);
  } else if ((int)blockIdx.x < a.ntiles) {
    stage_layer(0, 0);
  }
  // Before layer l of `tile` runs (non-resident): request the next layer.
  auto stage_next = [&](int l, int tile) {
    if (l + 1 < L) stage_layer(l + 1, step + 1);
    else if (tile + G < a.ntiles) stage_layer(0, step + 1);
  };
  // A_1 = X of a wave tile, in input order: lane group g takes features
  // 32 kb + 8 g .. + 7.
  // With VEC (in_dim a multiple of 8) each lane reads 16-byte pieces.
  auto load_x_t = [&](auto VECc, int tile, u32x4 (&dst)[NT][KBW]) {
    const int64_t r0 = (((int64_t)tile * NW + wave) * NT) * 16;
    int64_t vr = M - r0;
    vr = vr < 0 ? 0 : (vr > NT * 16 ? NT * 16 : vr);
    if constexpr (decltype(VECc)::value) {
      // per-lane byte offset inside a 16-row block; the block goes in the
      // scalar offset
      const rsrc_t xr = make_rsrc(a.X + r0 * in_dim, vr * in_dim * 2);
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) {
        const int f0 = kb * 32 + lg * 8;
        const uint32_t voff = (kb < KB0 && f0 < in_dim) ? (uint32_t)((li * in_dim + f0) * 2) : kOOB;
#pragma unroll
        for (int n = 0; n < NT; ++n) dst[n][kb] = bload128(xr, voff, (uint32_t)(n * 32 * in_dim));
      }
    } else {
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const int64_t m = r0 + n * 16 + li;
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
          const int f0 = kb * 32 + lg * 8;
          uint32_t e[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
          if (kb < KB0 && m < M && f0 < in_dim) {
            const uint16_t* xp = a.X + m * in_dim + f0;
#pragma unroll
            for (int q = 0; q < 8; ++q) e[q] = (f0 + q < in_dim) ? (uint32_t)xp[q] : 0u;
          }
          dst[n][kb] = u32x4{e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16),
                             e[6] | (e[7] << 16)};
        }
      }
    }
  };
  auto load_x = [&](int tile, u32x4 (&dst)[NT][KBW]) {
    if (xvec) load_x_t(std::true_type{}, tile, dst);
    else load_x_t(std::false_type{}, tile, dst);
  };
  auto load_xv = [&](int tile, u32x4 (&dst)[NT][KBW]) { load_x_t(std::true_type{}, tile, dst); };
  // Narrow nets have registers to spare for the X of later tiles: each
  // wave requests X two tiles ahead (two buffers, used in turn by a tile
  // loop unrolled by two).
  constexpr bool XPF = W <= 32;
  // Wider inference nets whose layers are all resident and whose output is
  // one 16-column strip run the last hidden layer and the output layer
  // together: each k-block of A_{L-1} enters the output product as soon as
  // its two strips exist, so A_{L-1} is never held whole and the second
  // activation buffer is free during those two layers.  The next tile's X
  // is requested into it there, hidden behind that work.
  // The launcher picks FU 1 or 2 only for inference with every layer
  // resident, L >= 2, SO == 1 and in_dim a multiple of 8.
  // Other inference nets of these widths (FU 3, 4; L >= 2, in_dim a
  // multiple of 8) keep the layers apart, and the next tile's X is
  // requested into the activation buffer the output layer does not read,
  // hidden behind that layer.
  constexpr bool FUSE = FU == 1 || FU == 2;
  constexpr bool OXP = FU == 3 || FU == 4;
  static_assert(FU == 0 || (!XPF && MODE == FWD_INFER), "early X fetch: W >= 64, inference");
  u32x4 xq0[XPF ? NT : 1][KBW], xq1[XPF ? NT : 1][KBW];
  u32x4 actA[NT][KBW], actB[NT][KBW];
  if constexpr (XPF) {
    if ((int)blockIdx.x < a.ntiles) load_x(blockIdx.x, xq0);
    if ((int)blockIdx.x + G < a.ntiles) load_x(blockIdx.x + G, xq1);
  } else if constexpr (FUSE || OXP) {
    if ((int)blockIdx.x < a.ntiles) load_xv(blockIdx.x, actA);
  }
  drain_and_sync();  // weights (the first layer, when streaming) in LDS

  // bf16(sigma(c)) of one 16-row block's four features, as two bf16 pairs.
  auto hid_act = [&](const f32x4& c, uint32_t& p0, uint32_t& p1) {
    if constexpr (ACT == ACT_RELU) {
      p0 = relu_bf16x2(pack_bf16x2(c[0], c[1]));
      p1 = relu_bf16x2(pack_bf16x2(c[2], c[3]));
    } else {
      p0 = pack_bf16x2(act_hidden<ACT>(c[0]), act_hidden<ACT>(c[1]));
      p1 = pack_bf16x2(act_hidden<ACT>(c[2]), act_hidden<ACT>(c[3]));
    }
  };

  float loss = 0.f;
  // One wave tile, with activation buffers bx (holding X) and by.  With F
  // its X is already in bx (requested by the previous tile or before the
  // loop); otherwise it comes from xq (XPF) or is loaded here.
  auto tile_body = [&](int tile, u32x4 (&bx)[NT][KBW], u32x4 (&by)[NT][KBW], auto Fc,
                       u32x4 (&xq)[XPF ? NT : 1][KBW]) {
    constexpr bool F = decltype(Fc)::value;
    const int64_t tb0 = ((int64_t)tile * NW + wave) * NT;  // first 16-row block
    const int64_t row0 = tb0 * 16;
    int64_t vrows = M - row0;  // valid rows of this wave's tile
    vrows = vrows < 0 ? 0 : (vrows > NT * 16 ? NT * 16 : vrows);
    const int vblk = (int)((vrows + 15) / 16);

    // Two activation buffers and two weight-fragment buffers, used in turn
    // (hidden layers go in pairs), so no register array is ever copied.
    u32x4 afb[2][KBW];
    if (resident && L > 1) load_frags<KBW>(smem, 0, lane, afb[0]);
    if constexpr (XPF) {
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) bx[n][kb] = xq[n][kb];
      if (tile + 2 * G < a.ntiles) load_x(tile + 2 * G, xq);
    } else if constexpr (!F && !OXP) {
      load_x(tile, bx);
    }

    // Hidden layer l: out = bf16(sigma(in W_l)) in the next layer's chain
    // order (see common.h).  P is the layer's parity within its pair; the
    // fragment buffer of strip s is (P * SW + s) % 2.
    auto hidden = [&](auto Pc, int l, const u32x4 (&in)[NT][KBW], u32x4 (&out)[NT][KBW]) {
      constexpr int P = decltype(Pc)::value;
      const u32x4* wl;
      if (resident) {
        wl = smem + (size_t)layer_off(l) * 64;
      } else {
        wl = stream_buf(step);
        stage_next(l, tile);
        load_frags<KBW>(wl, 0, lane, afb[(P * SW) & 1]);
      }
      const size_t soff = (size_t)l * a.M16 * W + (size_t)row0 * W;
      const rsrc_t sa = make_rsrc(a.stashA + soff, a.stashA ? (int64_t)vblk * 32 * W : 0);
      const rsrc_t ss = make_rsrc(a.stashS + soff, a.stashS ? (int64_t)vblk * 32 * W : 0);
      // ReLU mask words of this layer's activation (training, ReLU nets)
      constexpr bool MASK = MODE != FWD_INFER && ACT == ACT_RELU;
      uint32_t mk[NT];
#pragma unroll
      for (int n = 0; n < NT; ++n) mk[n] = 0u;
      if constexpr (SW == 1) {
        // width 16: the second half of the only k-block is padding
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          out[n][0].z = 0u;
          out[n][0].w = 0u;
        }
      }
      static_for<0, SW>([&](auto sc) {
        constexpr int s = decltype(sc)::value;
        constexpr int cur = (P * SW + s) & 1;
        if constexpr (s + 1 < SW) {
          load_frags<KBW>(wl, s + 1, lane, afb[cur ^ 1]);
        } else {
          if (resident && l + 1 < L - 1)
            load_frags<KBW>(smem + (size_t)layer_off(l + 1) * 64, 0, lane, afb[cur ^ 1]);
        }
        f32x4 acc[NT];
        strip_product<NT, KBW>(afb[cur], in, acc);
        u32x2 pq[TST ? NT : 1];
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          uint32_t p0, p1;
          hid_act(acc[n], p0, p1);
          pin(p0);
          pin(p1);
          if constexpr (s & 1) {
            out[n][s >> 1].z = p0;
            out[n][s >> 1].w = p1;
          } else {
            out[n][s >> 1].x = p0;
            out[n][s >> 1].y = p1;
          }
          if constexpr (MASK) {
            mk[n] |= (nonzero_halves(p0) | (nonzero_halves(p1) << 1)) << (2 * s);
            pin(mk[n]);
          }
          if constexpr (TST) {
            pq[n] = u32x2{p0, p1};
          } else if constexpr (MODE != FWD_INFER) {
            const uint32_t so = (uint32_t)((n * SW + s) * 512);
            bstore64<NTS>(u32x2{p0, p1}, sa, lane * 8, so);
            if constexpr (ACT == ACT_SINE) {
              const uint32_t c0 = pack_bf16x2(__cosf(acc[n][0]), __cosf(acc[n][1]));
              const uint32_t c1 = pack_bf16x2(__cosf(acc[n][2]), __cosf(acc[n][3]));
              bstore64<NTS>(u32x2{c0, c1}, ss, lane * 8, so);
            }
          }
        }
        if constexpr (TST) {
          // the strip of blocks n, n + 1 transposed, each into its own 512
          // bytes (rows past M are dropped by the range check as above)
#pragma unroll
          for (int n = 0; n < NT; n += 2) {
            const u32x4 src = {pq[n].x, pq[n].y, pq[n + 1].x, pq[n + 1].y};
            const f32x4 o0 = mfma16(src, sel0, zero4), o1 = mfma16(src, sel1, zero4);
            bstore64<NTS>(u32x2{pack_bf16x2(o0[0], o0[1]), pack_bf16x2(o0[2], o0[3])}, sa, lane * 8,
                          (uint32_t)((n * SW + s) * 512));
            bstore64<NTS>(u32x2{pack_bf16x2(o1[0], o1[1]), pack_bf16x2(o1[2], o1[3])}, sa, lane * 8,
                          (uint32_t)(((n + 1) * SW + s) * 512));
          }
        }
        // Keep each strip's work together: bounds the live registers.
        __builtin_amdgcn_sched_barrier(0);
      });
      if constexpr (MASK) {
        const rsrc_t mr = make_rsrc(a.reluMask + ((size_t)l * (a.M16 / 16) + tb0) * 64,
                                    a.reluMask ? (int64_t)vblk * 256 : 0);
#pragma unroll
        for (int n = 0; n < NT; ++n) bstore32<NTS>(mk[n], mr, lane * 4, (uint32_t)(n * 256));
      }
      if (!resident) {
        drain_and_sync();  // next layer staged; this buffer free again
        ++step;
      }
    };

    // Everything after the product of output strip s: Y = sigma_out(C_L);
    // when training also the loss and the output delta
    // 2 (Y - T) / (M out_dim) * sigma_out'(C_L); when stashing C_L.
    auto out_strip = [&](int s, const f32x4 (&acc)[NT]) {
      const rsrc_t yr = make_rsrc(a.Y + row0 * out_dim, a.Y ? vrows * out_dim * 2 : 0);
      const int j0 = s * 16 + lg * 4;
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const int64_t m = row0 + n * 16 + li;
        const bool ok = (m < M) && (j0 < out_dim);
        // element offset of (row li, j0) inside the block (past the end if
        // the column is); the block's offset goes in the scalar offset
        const uint32_t eo = (j0 < out_dim) ? (uint32_t)(li * out_dim + j0) : kOOB / 4;
        const uint32_t bo = (uint32_t)(n * 16 * out_dim);
        float y[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) y[r] = act_apply(out_act, acc[n][r]);
        const uint32_t y0 = pack_bf16x2(y[0], y[1]), y1 = pack_bf16x2(y[2], y[3]);
        if (a.Y != nullptr) {
          if (yvec) {
            // Y rows wider than one strip are completed by several stores,
            // which the caches must merge: inference stores them with the
            // default policy then (measured: width 64, out 64, 189 -> 80 us
            // at 2^20 rows).
            if (MODE == FWD_INFER && NTS && SO == 1)
              bstore64<true>(u32x2{y0, y1}, yr, eo * 2, bo * 2);
            else
              bstore64<NTS && MODE != FWD_INFER>(u32x2{y0, y1}, yr, eo * 2, bo * 2);
          } else if (ok) {
            uint16_t* yp = a.Y + m * out_dim + j0;
            const uint16_t yb[4] = {(uint16_t)(y0 & 0xffff), (uint16_t)(y0 >> 16),
                                    (uint16_t)(y1 & 0xffff), (uint16_t)(y1 >> 16)};
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (j0 + r < out_dim) yp[r] = yb[r];
          }
        }
        if constexpr (MODE == FWD_TRAIN) {
          const rsrc_t tr = make_rsrc(a.T + row0 * out_dim, a.T ? vrows * out_dim * 4 : 0);
          const rsrc_t dr = make_rsrc(a.deltaOut + row0 * OP, a.deltaOut ? (int64_t)vblk * 32 * OP : 0);
          float t[4] = {0.f, 0.f, 0.f, 0.f};
          if (yvec) {
            const u32x4 tv = bload128(tr, eo * 4, bo * 4);
            t[0] = __uint_as_float(tv.x);
            t[1] = __uint_as_float(tv.y);
            t[2] = __uint_as_float(tv.z);
            t[3] = __uint_as_float(tv.w);
          } else if (ok) {
            const float* tp = a.T + m * out_dim + j0;
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (j0 + r < out_dim) t[r] = tp[r];
          }
          float d[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const bool valid = ok && (j0 + r < out_dim);
            const float diff = y[r] - t[r];
            if (valid) loss += diff * diff;
            d[r] = valid ? (a.scale * diff) * act_out_grad(out_act, acc[n][r], y[r]) : 0.f;
          }
          bstore64<NTS>(u32x2{pack_bf16x2(d[0], d[1]), pack_bf16x2(d[2], d[3])}, dr, lane * 8,
                   (uint32_t)((n * SO + s) * 512));
        }
        if constexpr (MODE == FWD_STASH) {
          const rsrc_t cr = make_rsrc(a.cOut + row0 * OP, a.cOut ? (int64_t)vblk * 64 * OP : 0);
          bstore128<NTS>(__builtin_bit_cast(u32x4, acc[n]), cr, lane * 16,
                    (uint32_t)((n * SO + s) * 1024));
        }
      }
    };

    // Output layer on its own; with OXP the next tile's X goes to nx.
    auto output = [&](const u32x4 (&in)[NT][KBW], u32x4 (&nx)[NT][KBW]) {
      const int l = L - 1;
      const u32x4* wl;
      if (resident) {
        wl = smem + (size_t)layer_off(l) * 64;
      } else {
        wl = stream_buf(step);
        stage_next(l, tile);
      }
      if constexpr (OXP) {
        if (tile + G < a.ntiles) load_xv(tile + G, nx);
      }
      for (int s = 0; s < SO; ++s) {
        u32x4 af[KBW];
        load_frags<KBW>(wl, s, lane, af);
        f32x4 acc[NT];
        strip_product<NT, KBW>(af, in, acc);
        out_strip(s, acc);
      }
      if (!resident) {
        drain_and_sync();
        ++step;
      }
    };

    // Last hidden layer (L - 2) and the one-strip output layer together
    // (F only; every layer resident, SW even).  `nx` is free throughout:
    // the next tile's X goes there.
    auto last = [&](const u32x4 (&in)[NT][KBW], u32x4 (&nx)[NT][KBW]) {
      const u32x4* wl = smem + (size_t)layer_off(L - 2) * 64;
      const u32x4* wo = smem + (size_t)layer_off(L - 1) * 64;
      if (tile + G < a.ntiles) load_xv(tile + G, nx);
      f32x4 yacc[NT];
#pragma unroll
      for (int n = 0; n < NT; ++n) yacc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
      u32x4 kblk[NT];  // one k-block of A_{L-1}: strips 2 kb and 2 kb + 1
      u32x4 wof;       // the output layer's fragment for that k-block
      static_for<0, SW>([&](auto sc) {
        constexpr int s = decltype(sc)::value;
        constexpr int cur = s & 1;
        if constexpr (s + 1 < SW) load_frags<KBW>(wl, s + 1, lane, afb[cur ^ 1]);
        if constexpr ((s & 1) == 0) wof = wo[(s >> 1) * 64 + lane];
        f32x4 acc[NT];
        strip_product<NT, KBW>(afb[cur], in, acc);
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          uint32_t p0, p1;
          hid_act(acc[n], p0, p1);
          pin(p0);
          pin(p1);
          if constexpr (s & 1) {
            kblk[n].z = p0;
            kblk[n].w = p1;
          } else {
            kblk[n].x = p0;
            kblk[n].y = p1;
          }
        }
        // the same k-block order and MFMA shape as the output layer on its
        // own, so Y is bitwise the same as the training forward's
        if constexpr (s & 1) {
#pragma unroll
          for (int n = 0; n < NT; ++n) yacc[n] = mfma16(wof, kblk[n], yacc[n]);
        }
        __builtin_amdgcn_sched_barrier(0);
      });
      out_strip(0, yacc);
    };

    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    int l = 0;
    if constexpr (F) {
      static_assert(SW % 2 == 0, "fused last layers need an even strip count");
      for (; l + 2 <= L - 2; l += 2) {
        hidden(I0{}, l, bx, by);
        hidden(I1{}, l + 1, by, bx);
      }
      if (l < L - 2) {
        hidden(I0{}, l, bx, by);
        last(by, bx);
      } else {
        last(bx, by);
      }
    } else {
      for (; l + 2 <= L - 1; l += 2) {
        hidden(I0{}, l, bx, by);
        hidden(I1{}, l + 1, by, bx);
      }
      if (l < L - 1) {
        hidden(I0{}, l, bx, by);
        output(by, bx);
      } else {
        output(bx, by);
      }
    }
  };

  using NoF = std::integral_constant<bool, false>;
  if constexpr (XPF) {
    for (int tile = blockIdx.x; tile < a.ntiles; tile += 2 * G) {
      tile_body(tile, actA, actB, NoF{}, xq0);
      if (tile + G < a.ntiles) tile_body(tile + G, actA, actB, NoF{}, xq1);
    }
  } else if constexpr (FU == 2) {
    // The last layers read A_{L-1} from the buffer the hidden chain ends
    // in and the next X goes to the other one; with L even that is actB
    // after a tile that started in actA and the reverse, so the loop
    // alternates.
    using Fu = std::integral_constant<bool, true>;
    for (int tile = blockIdx.x; tile < a.ntiles; tile += 2 * G) {
      tile_body(tile, actA, actB, Fu{}, xq0);
      if (tile + G < a.ntiles) tile_body(tile + G, actB, actA, Fu{}, xq0);
    }
  } else if constexpr (FU == 1) {
    using Fu = std::integral_constant<bool, true>;
    for (int tile = blockIdx.x; tile < a.ntiles; tile += G) tile_body(tile, actA, actB, Fu{}, xq0);
  } else if constexpr (FU == 4) {
    // L odd: the output layer reads the buffer the tile started in, so the
    // next X lands in the other one and the loop alternates.
    for (int tile = blockIdx.x; tile < a.ntiles; tile += 2 * G) {
      tile_body(tile, actA, actB, NoF{}, xq0);
      if (tile + G < a.ntiles) tile_body(tile + G, actB, actA, NoF{}, xq0);
    }
  } else {
    for (int tile = blockIdx.x; tile < a.ntiles; tile += G) tile_body(tile, actA, actB, NoF{}, xq0);
  }

  if constexpr (MODE == FWD_TRAIN) {
    const float v = wave_sum(loss);
    // The weights are no longer read (and no layer is being staged after
    // the last tile): the per-wave sums go into the start of that LDS, so
    // the kernel has no static LDS and all of it can hold weights.
    __syncthreads();
    float* red = reinterpret_cast<float*>(smem);
    if (lane == 0) red[wave] = v;
    __syncthreads();
    if (tid == 0) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) s += red[w];
      a.lossPart[blockIdx.x] = s;
    }
  }
}

// A kernel instantiation with its block size and row tile.
struct FwdPick {
  void (*kern)(FwdArgs);
  int threads;
  int64_t rows;
};
template <int W, int ACT, int MODE, int FU, bool RES, bool SMALL = false, bool LIN = false, bool TST = false>
static FwdPick fwd_pick() {
  constexpr int NW = fwd_waves<W, MODE, SMALL, FU>(), NT = fwd_nt<W, MODE, SMALL, FU>();
  return FwdPick{fwd_kernel<W, ACT, MODE, FU, RES, SMALL, LIN, TST>, NW * 64, (int64_t)NW * NT * 16};
}

// LIN: the output activation is linear (the common case) and fixed at
// compile time.  With a runtime output activation the epilogue switches per
// element, which cost 12% of width-16 inference at 2^20 rows (17.9 -> 15.7
// us) and 1-2% at the other widths.
template <int W, int ACT, int MODE, bool LIN>
static hipError_t launch_t(const FwdArgs& a0, hipStream_t stream, int* grid_out) {
  FwdArgs a = a0;
  DeviceInfo di;
  hipError_t e = device_info(&di);
  if (e != hipSuccess) return e;
  const int KBW = (W + 31) / 32, SW = W / 16;
  const int SO = (a.out_dim + 15) / 16;
  const uint32_t maxf = (uint32_t)((a.L > 1 ? SW : SO) * KBW);
  const size_t res_bytes = (size_t)a.total_frags * 1024;
  // The kernel has no static LDS, so inference keeps weights that fill all
  // of it resident (width 128, out 128, 5 matrices: 227 -> 194 us at 2^20
  // rows); the training forward of such a net measured faster streamed
  // (1297 against 1334 us for the whole step), so it keeps 1 KiB spare.
  a.resident = res_bytes + (MODE == FWD_INFER ? 0 : 1024) <= (size_t)di.max_lds ? 1 : 0;
  const size_t lds = a.resident ? res_bytes : (size_t)2 * maxf * 1024;
  FwdPick pk = a.resident ? fwd_pick<W, ACT, MODE, 0, true, false, LIN>() : fwd_pick<W, ACT, MODE, 0, false, false, LIN>();
  if constexpr (W == 128 && MODE == FWD_TRAIN) {
    if (a.stash_t)
      pk = a.resident ? fwd_pick<W, ACT, MODE, 0, true, false, LIN, true>()
                      : fwd_pick<W, ACT, MODE, 0, false, false, LIN, true>();
  } else {
    if (a.stash_t) return hipErrorInvalidValue;  // only the width-128 training forward writes it
  }
  if constexpr (MODE == FWD_INFER && W >= 64) {
    if (a.resident && a.L >= 2 && SO == 1 && (a.in_dim % 8) == 0)
      pk = (a.L & 1) ? fwd_pick<W, ACT, MODE, 1, true, false, LIN>() : fwd_pick<W, ACT, MODE, 2, true, false, LIN>();
    else if (a.L >= 2 && (a.in_dim % 8) == 0)
      pk = a.resident ? ((a.L & 1) ? fwd_pick<W, ACT, MODE, 4, true, false, LIN>()
                                   : fwd_pick<W, ACT, MODE, 3, true, false, LIN>())
                      : ((a.L & 1) ? fwd_pick<W, ACT, MODE, 4, false, false, LIN>()
                                   : fwd_pick<W, ACT, MODE, 3, false, false, LIN>());
  }
  if constexpr (W <= 64) {
    // Small batches: fewer than two row tiles of the tile configuration
    // (NT NW 16 rows) per CU (widths up to 64, whose weights leave LDS for
    // several workgroups per CU), inference and training forward alike.
    const int64_t cfg_rows = (int64_t)TileCfg<W>::NT * TileCfg<W>::NW * 16;
    if ((a.M + cfg_rows - 1) / cfg_rows <= 2 * (int64_t)di.cus && a.resident)
      pk = fwd_pick<W, ACT, MODE, 0, true, true, LIN>();
  }
  a.ntiles = (int)((a.M + pk.rows - 1) / pk.rows);
  int occ = 0;
  e = kernel_occupancy(reinterpret_cast<const void*>(pk.kern), pk.threads, lds, &occ);
  if (e != hipSuccess) return e;
  int grid = di.cus * occ;
  if (grid > a.ntiles) grid = a.ntiles;
  if (grid > kMaxLossParts) grid = kMaxLossParts;
  if (grid < 1) grid = 1;
  if (grid_out) *grid_out = grid;
  hipLaunchKernelGGL(pk.kern, dim3(grid), dim3(pk.threads), lds, stream, a);
  return hipGetLastError();
}

template <int W, int ACT>
static hipError_t by_mode(int mode, const FwdArgs& a, hipStream_t s, int* g) {
  switch (mode) {
    case FWD_INFER:
      return a.out_act == ACT_LINEAR ? launch_t<W, ACT, FWD_INFER, true>(a, s, g)
                                     : launch_t<W, ACT, FWD_INFER, false>(a, s, g);
    case FWD_STASH: return launch_t<W, ACT, FWD_STASH, false>(a, s, g);
    default:
      return a.out_act == ACT_LINEAR ? launch_t<W, ACT, FWD_TRAIN, true>(a, s, g)
                                     : launch_t<W, ACT, FWD_TRAIN, false>(a, s, g);
  }
}

template <int W>
static hipError_t by_act(int act, int mode, const FwdArgs& a, hipStream_t s, int* g) {
  switch (act) {
    case ACT_RELU: return by_mode<W, ACT_RELU>(mode, a, s, g);
    case ACT_SIGMOID: return by_mode<W, ACT_SIGMOID>(mode, a, s, g);
    case ACT_SINE: return by_mode<W, ACT_SINE>(mode, a, s, g);
    default: return by_mode<W, ACT_LINEAR>(mode, a, s, g);
  }
}

// Per-width entry points, each compiled in its own translation unit
// (fwd16.hip .. fwd128.hip) so the build runs in parallel; fwd.hip
// dispatches on the width.
template <int W>
hipError_t launch_forward_w(int act, int mode, const FwdArgs& a, hipStream_t s, int* grid_out);

}  // namespace ffmlp
