// Fused backward kernel: delta propagation of Algorithm 2 (arXiv 2403.17607,
// section III-A), D_i = sigma_b(A_i, D_{i+1} B_i^T) for i = nlayers-1 .. 2.
//
// Same structure as the forward kernel, walking the layers in reverse: the
// deltas of a wave's batch rows stay in VGPRs as MFMA B operands, the
// product D_l^T = W_l D_{l+1}^T uses the backward-packed (non-transposed)
// weights as the A operand, and the activation derivative is read from the
// stash the forward pass wrote.  Every delta is stored for the weight
// gradient kernel.  No delta of the input layer is formed (the algorithm
// stops at i = 2).
//
// Seeded mode (mlp_backward) builds the output delta from a caller-given
// dY and the stashed pre-activation of the output layer; otherwise the
// output delta written by the training forward pass is read back.
#pragma once

#include "device.h"

namespace ffmlp {

// RES: every layer's weights resident in LDS (else staged layer by layer);
// each mode is its own kernel, so the tile loop carries no residency
// branches (whose joins force conservative waits on LDS loads).
template <int W, int ACT, int SEEDED, bool RES, bool DX>
__global__ __launch_bounds__(TileCfg<W>::NW * 64) void bwd_kernel(const BwdArgs a) {
  constexpr int NT = TileCfg<W>::NT, NW = TileCfg<W>::NW;
  constexpr int KBW = (W + 31) / 32, SW = W / 16;
  extern __shared__ u32x4 smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int li = lane & 15, lg = lane >> 4;
  const int L = a.L, out_dim = a.out_dim, out_act = a.out_act;
  const int64_t M = a.M;
  const int SO = (out_dim + 15) >> 4;
  const int OP = SO * 16;
  const bool yvec = (out_dim & 3) == 0;

  // Weights: resident in LDS, or staged layer by layer through two LDS
  // buffers with direct-to-LDS loads, the next layer (layer L-1 of the next
  // tile after layer 1) loading while the current one computes.
  constexpr bool resident = RES;
  const int G = gridDim.x;
  const uint32_t bufq = (uint32_t)(SW * KBW) * 64;  // one buffer, in u32x4
  int step = 0;
  auto stream_buf = [&](int st) { return smem + ((st & 1) ? bufq : 0u); };
  auto stage_layer = [&](int l, int st) {
    stage_frags(stream_buf(st), a.packed + (size_t)(l - 1) * a.layH_frags * 64,
                (uint32_t)(SW * KBW), wave, NW, lane);
  };
  if (L > 1) {
    if (resident) {
      stage_frags(smem, a.packed, a.total_frags, wave, NW, lane);
    } else if ((int)blockIdx.x < a.ntiles) {
      stage_layer(L - 1, 0);
    }
    drain_and_sync();
  }
  for (int tile = blockIdx.x; tile < a.ntiles; tile += G) {
    const int64_t tb0 = ((int64_t)tile * NW + wave) * NT;
    const int64_t row0 = tb0 * 16;
    int64_t vrows = M - row0;  // valid rows of this wave's tile
    vrows = vrows < 0 ? 0 : (vrows > NT * 16 ? NT * 16 : vrows);
    const int vblk = (int)((vrows + 15) / 16);
    u32x4 dA[NT][KBW], dB[NT][KBW];
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) dA[n][kb] = u32x4{0u, 0u, 0u, 0u};

    // Output delta, in chain order.
    {
      const rsrc_t dr = make_rsrc(a.deltaOut + row0 * OP, (int64_t)vblk * 32 * OP);
      const rsrc_t cr = make_rsrc(a.cOut + row0 * OP, a.cOut ? (int64_t)vblk * 64 * OP : 0);
      const rsrc_t gr = make_rsrc(a.dY + row0 * out_dim, a.dY ? vrows * out_dim * 4 : 0);
      static_for<0, SW>([&](auto sc) {
        constexpr int s = decltype(sc)::value;
        if (s >= SO) return;
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          const uint32_t so = (uint32_t)((n * SO + s) * 512);
          uint32_t p0, p1;
          if constexpr (!SEEDED) {
            const u32x2 v = bload64(dr, lane * 8, so);
            p0 = v.x;
            p1 = v.y;
          } else {
            const int64_t m = row0 + n * 16 + li;
            const int j0 = s * 16 + lg * 4;
            const bool ok = m < M && j0 < out_dim;
            float g[4] = {0.f, 0.f, 0.f, 0.f};
            if (yvec) {
              const uint32_t eo = (j0 < out_dim) ? (uint32_t)(li * out_dim + j0) : kOOB / 4;
              const u32x4 v = bload128(gr, eo * 4, (uint32_t)(n * 64 * out_dim));
              g[0] = __uint_as_float(v.x);
              g[1] = __uint_as_float(v.y);
              g[2] = __uint_as_float(v.z);
              g[3] = __uint_as_float(v.w);
            } else if (ok) {
              const float* dp = a.dY + m * out_dim + j0;
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if (j0 + r < out_dim) g[r] = dp[r];
            }
            if (out_act != ACT_LINEAR) {
              const u32x4 cv = bload128(cr, lane * 16, (uint32_t)((n * SO + s) * 1024));
              const float c[4] = {__uint_as_float(cv.x), __uint_as_float(cv.y),
                                  __uint_as_float(cv.z), __uint_as_float(cv.w)};
#pragma unroll
              for (int r = 0; r < 4; ++r) g[r] *= act_out_grad(out_act, c[r], act_apply(out_act, c[r]));
            }
            p0 = pack_bf16x2(g[0], g[1]);
            p1 = pack_bf16x2(g[2], g[3]);
            bstore64(u32x2{p0, p1}, dr, lane * 8, so);
          }
          if (s & 1) {
            dA[n][s >> 1].z = p0;
            dA[n][s >> 1].w = p1;
          } else {
            dA[n][s >> 1].x = p0;
            dA[n][s >> 1].y = p1;
          }
        }
      });
    }

    // ReLU: the mask words of the activation a layer needs (stash index
    // l - 1 for layer l), requested one layer ahead.
    const size_t mblk = (size_t)(a.M16 / 16);
    auto mask_rsrc = [&](int idx) {
      return make_rsrc(a.reluMask + ((size_t)idx * mblk + tb0) * 64, a.reluMask ? (int64_t)vblk * 256 : 0);
    };
    uint32_t mw[NT];
    if constexpr (ACT == ACT_RELU) {
      if (L > 1) {
        const rsrc_t mr = mask_rsrc(L - 2);
#pragma unroll
        for (int n = 0; n < NT; ++n) mw[n] = bload32(mr, lane * 4, (uint32_t)(n * 256));
      }
    }

    // Backward layer l: out = bf16((in W_l^T) * sigma'(a_l)), the delta of
    // layer l-1 in chain order; it is also stored for the gradient kernel.
    // The derivative source of strip s is requested PF strips ahead (ReLU:
    // the layer's mask words, requested during the previous layer).
    auto layer = [&](int l, const u32x4 (&in)[NT][KBW], u32x4 (&out)[NT][KBW]) {
      const u32x4* wl;
      if (resident) {
        wl = smem + (size_t)(l - 1) * a.layH_frags * 64;
      } else {
        wl = stream_buf(step);
        if (l - 1 >= 1) stage_layer(l - 1, step + 1);
        else if (tile + G < a.ntiles) stage_layer(L - 1, step + 1);
      }
      const size_t toff = (size_t)(l - 1) * a.M16 * W + (size_t)row0 * W;
      const rsrc_t gsrc = make_rsrc((ACT == ACT_SINE ? a.stashS : a.stashA) + toff, (int64_t)vblk * 32 * W);
      const rsrc_t dst = make_rsrc(a.deltaH + toff, (int64_t)vblk * 32 * W);
      if constexpr (SW == 1) {
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          out[n][0].z = 0u;
          out[n][0].w = 0u;
        }
      }
      constexpr int PF = SW < 4 ? SW : 4;
      u32x2 gv[SW][NT];
      uint32_t mwn[NT];
      if constexpr (ACT == ACT_RELU) {
        if (l - 1 >= 1) {
          const rsrc_t mr = mask_rsrc(l - 2);
#pragma unroll
          for (int n = 0; n < NT; ++n) mwn[n] = bload32(mr, lane * 4, (uint32_t)(n * 256));
        }
      }
      auto request = [&](int s) {
        if constexpr (ACT != ACT_LINEAR && ACT != ACT_RELU) {
#pragma unroll
          for (int n = 0; n < NT; ++n) gv[s][n] = bload64(gsrc, lane * 8, (uint32_t)((n * SW + s) * 512));
        }
      };
      static_for<0, PF>([&](auto sc) { request(decltype(sc)::value); });

      static_for<0, SW>([&](auto sc) {
        constexpr int s = decltype(sc)::value;
        if constexpr (s + PF < SW) request(s + PF);
        // every packed layer has KBW k-blocks (the output layer's are
        // zero-padded past out_dim)
        u32x4 af[KBW];
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) af[kb] = wl[(s * KBW + kb) * 64 + lane];
        f32x4 acc[NT];
#pragma unroll
        for (int n = 0; n < NT; ++n) acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb)
#pragma unroll
          for (int n = 0; n < NT; ++n) acc[n] = mfma16(af[kb], in[n][kb], acc[n]);
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          uint32_t p0, p1;
          if constexpr (ACT == ACT_RELU) {
            // relu'(a) is [a > 0]; zero the rounded products where a is 0
            const uint32_t t = mw[n] >> (2 * s);
            p0 = mask_halves(pack_bf16x2(acc[n][0], acc[n][1]), t & 0x00010001u);
            p1 = mask_halves(pack_bf16x2(acc[n][2], acc[n][3]), (t >> 1) & 0x00010001u);
          } else if constexpr (ACT == ACT_LINEAR) {
            p0 = pack_bf16x2(acc[n][0], acc[n][1]);
            p1 = pack_bf16x2(acc[n][2], acc[n][3]);
          } else {
            p0 = pack_bf16x2(acc[n][0] * act_hidden_grad<ACT>(bf16_lo(gv[s][n].x)),
                             acc[n][1] * act_hidden_grad<ACT>(bf16_hi(gv[s][n].x)));
            p1 = pack_bf16x2(acc[n][2] * act_hidden_grad<ACT>(bf16_lo(gv[s][n].y)),
                             acc[n][3] * act_hidden_grad<ACT>(bf16_hi(gv[s][n].y)));
          }
          if constexpr (s & 1) {
            out[n][s >> 1].z = p0;
            out[n][s >> 1].w = p1;
          } else {
            out[n][s >> 1].x = p0;
            out[n][s >> 1].y = p1;
          }
          bstore64(u32x2{p0, p1}, dst, lane * 8, (uint32_t)((n * SW + s) * 512));
        }
        // Keep each strip's work together: bounds the live registers.
        __builtin_amdgcn_sched_barrier(0);
      });
      if constexpr (ACT == ACT_RELU) {
#pragma unroll
        for (int n = 0; n < NT; ++n) mw[n] = mwn[n];
      }
      if (!resident) {
        drain_and_sync();  // next layer staged; this buffer free again
        ++step;
      }
    };

    // Input gradient (DX; an extension beyond Algorithm 2): dX^T = W_1 D_1^T
    // (1-based), no activation derivative, fp32 out.  The backward-packed
    // first layer is read straight from global memory (L2), not from LDS:
    // it is needed once per tile and would push the resident set past LDS.
    auto input_grad = [&](const u32x4 (&in)[NT][KBW]) {
      const int in_dim = a.in_dim;
      const int SI = (in_dim + 15) >> 4;
      const bool xv = (in_dim & 3) == 0;
      const rsrc_t xr = make_rsrc(a.dX + row0 * in_dim, vrows * in_dim * 4);
      // strip s + 1's fragments are requested while strip s computes
      u32x4 af[KBW], an[KBW];
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) an[kb] = a.packed0[kb * 64 + lane];
      for (int s = 0; s < SI; ++s) {
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) af[kb] = an[kb];
        if (s + 1 < SI) {
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb) an[kb] = a.packed0[((s + 1) * KBW + kb) * 64 + lane];
        }
        f32x4 acc[NT];
#pragma unroll
        for (int n = 0; n < NT; ++n) acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb)
#pragma unroll
          for (int n = 0; n < NT; ++n) acc[n] = mfma16(af[kb], in[n][kb], acc[n]);
        const int f0 = 16 * s + 4 * lg;
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          if (xv) {
            const uint32_t eo = f0 < in_dim ? (uint32_t)((li * in_dim + f0) * 4) : kOOB;
            bstore128(__builtin_bit_cast(u32x4, acc[n]), xr, eo, (uint32_t)(n * 16 * in_dim * 4));
          } else {
            const int64_t m = row0 + n * 16 + li;
            if (m < M) {
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if (f0 + r < in_dim) a.dX[m * in_dim + f0 + r] = acc[n][r];
            }
          }
        }
      }
    };

    // Layers in pairs with two delta buffers, so no register array is copied.
    int l = L - 1;
    for (; l - 2 >= 0; l -= 2) {
      layer(l, dA, dB);
      layer(l - 1, dB, dA);
    }
    if (l >= 1) {
      layer(l, dA, dB);
      if constexpr (DX) input_grad(dB);
    } else {
      if constexpr (DX) input_grad(dA);
    }
  }
}

template <int W, int ACT, int SEEDED>
static hipError_t launch_t(const BwdArgs& a0, hipStream_t stream) {
  constexpr int NTH = TileCfg<W>::NW * 64;
  BwdArgs a = a0;
  DeviceInfo di;
  hipError_t e = device_info(&di);
  if (e != hipSuccess) return e;
  const size_t res_bytes = (size_t)a.total_frags * 1024;
  a.resident = res_bytes <= (size_t)di.max_lds ? 1 : 0;  // the kernel has no static LDS
  size_t lds = a.resident ? res_bytes : (size_t)2 * a.layH_frags * 1024;
  if (lds == 0) lds = 16;
  auto kern = a.resident ? bwd_kernel<W, ACT, SEEDED, true, false> : bwd_kernel<W, ACT, SEEDED, false, false>;
  if constexpr (SEEDED) {
    if (a.dX != nullptr)
      kern = a.resident ? bwd_kernel<W, ACT, SEEDED, true, true> : bwd_kernel<W, ACT, SEEDED, false, true>;
  }
  int occ = 0;
  e = kernel_occupancy(reinterpret_cast<const void*>(kern), NTH, lds, &occ);
  if (e != hipSuccess) return e;
  int grid = di.cus * occ;
  if (grid > a.ntiles) grid = a.ntiles;
  if (grid < 1) grid = 1;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(NTH), lds, stream, a);
  return hipGetLastError();
}

template <int W, int ACT>
static hipError_t by_seed(int seeded, const BwdArgs& a, hipStream_t s) {
  return seeded ? launch_t<W, ACT, 1>(a, s) : launch_t<W, ACT, 0>(a, s);
}

template <int W>
static hipError_t by_act(int act, int seeded, const BwdArgs& a, hipStream_t s) {
  switch (act) {
    case ACT_RELU: return by_seed<W, ACT_RELU>(seeded, a, s);
    case ACT_SIGMOID: return by_seed<W, ACT_SIGMOID>(seeded, a, s);
    case ACT_SINE: return by_seed<W, ACT_SINE>(seeded, a, s);
    default: return by_seed<W, ACT_LINEAR>(seeded, a, s);
  }
}

// Per-width entry points, each compiled in its own translation unit
// (bwd16.hip .. bwd128.hip); bwd.hip dispatches on the width.
template <int W>
hipError_t launch_backward_w(int act, int seeded, const BwdArgs& a, hipStream_t s);

}  // namespace ffmlp
