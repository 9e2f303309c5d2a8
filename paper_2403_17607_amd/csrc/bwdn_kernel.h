// Fused backward pass with the weight gradients for widths 16 and 32: the
// delta loop of Algorithm 2 and G_i = A_i^T D_{i+1} (arXiv 2403.17607,
// section III-A; fusing G into the backward pass is the paper's future work,
// section V) in one kernel with no exchange between waves.
//
// At these widths a whole layer's G is one (width 16) or four (width 32)
// 16x16 tiles, so every wave keeps all layers' G in registers and contracts
// over its own rows only: no delta tile in LDS and no barrier in the tile
// loop.  Each wave owns NT 16-row blocks of a tile:
//   - the deltas of its rows stay in VGPRs (chain order) and go through the
//     layers in reverse, with the backward-packed weights resident in LDS as
//     the MFMA A operand;
//   - for each layer it loads the stashed activations of its rows (or X),
//     which serve both as the ReLU / sigmoid derivative source and as the
//     contraction operand of G;
//   - both contraction operands are transposed on the matrix cores (an MFMA
//     against a 0/1 selection matrix, exact) so that each lane holds 8 batch
//     rows of one feature, and G accumulates in fp32.
// At the end the waves add their G in a fixed order through LDS, one layer
// at a time, and each workgroup writes one partial for the fixed-order
// reduce kernel.  The derivative source is the ReLU mask words (DER 0), the
// stored activations for ReLU (DER 1), or (DER 2) sigmoid a (1 - a) of the
// stored a, sine the stored cos, linear 1.
#pragma once

#include "device.h"

namespace ffmlp {

constexpr int kBwdnWaves = 8, kBwdnNT = 4;  // 8 waves x 4 blocks: 512-row tiles
constexpr int kBwdnRows = kBwdnWaves * kBwdnNT * 16;

template <int W, int L, int OS>
struct BwdnGeom {
  static constexpr int SW = W / 16, KBW = (W + 31) / 32;
  static constexpr int KBO = (OS * 16 + 31) / 32;
  static constexpr int WFRAGS = (L - 2) * SW * KBW + SW * KBO;
  static constexpr int woff(int l) { return (l - 1) * SW * KBW; }
  static constexpr int sd(int l) { return l == L - 1 ? OS : SW; }  // j strips of G_l
  static constexpr int goff(int l) {  // first accumulator of G_l: SW x sd tiles
    int o = 0;
    for (int i = 0; i < l; ++i) o += SW * sd(i);
    return o;
  }
  static constexpr int nacc() { return goff(L); }
  // LDS: the weights, then one layer's G of every wave for the final sum.
  static constexpr size_t red_floats() { return (size_t)kBwdnWaves * W * W; }
  static constexpr size_t lds_bytes() { return (size_t)WFRAGS * 1024 + red_floats() * 4; }
  static_assert(W <= 32 && L >= 2 && L <= kBwdgMaxL && KBO <= KBW, "narrow fused backward");
};

template <int W, int L, int OS, int SEEDED, int DER>
__global__ __launch_bounds__(kBwdnWaves * 64) void bwdn_kernel(const BwdgArgs a) {
  using Gm = BwdnGeom<W, L, OS>;
  constexpr int NW = kBwdnWaves, NT = kBwdnNT, SW = Gm::SW, KBW = Gm::KBW, KBO = Gm::KBO;
  constexpr int NACC = Gm::nacc();
  constexpr int CSW = DER == 2 ? SW : 1;  // strips of the sine cos source
  extern __shared__ u32x4 smem[];
  float* red = reinterpret_cast<float*>(smem + (size_t)Gm::WFRAGS * 64);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int li = lane & 15, lg = lane >> 4;
  const int64_t M = a.M;
  const int in_dim = a.in_dim, out_dim = a.out_dim, act = a.act, out_act = a.out_act;
  const bool xvec = (in_dim & 3) == 0;
  const int SO = (out_dim + 15) >> 4;
  const int OP = SO * 16;
  const bool yvec = (out_dim & 3) == 0;

  // Resident weights: backward layers 1 .. L-2 whole, the output layer's
  // first KBO k-blocks of each strip.
  stage_frags(smem, a.packed, (uint32_t)((L - 2) * SW * KBW), wave, NW, lane);
  {
    const u32x4* src = a.packed + (size_t)(L - 2) * a.layH_frags * 64;
    u32x4* dst = smem + (size_t)Gm::woff(L - 1) * 64;
    for (int f = wave; f < SW * KBO; f += NW) {
      const int s = f / KBO, kb = f - s * KBO;
      __builtin_amdgcn_global_load_lds(
          (const void __attribute__((address_space(1)))*)(src + (size_t)(s * KBW + kb) * 64 + lane),
          (void __attribute__((address_space(3)))*)(dst + (size_t)f * 64), 16, 0, 0);
    }
  }
  // Selection matrices: an MFMA of an operand whose lane (g, i) holds row i
  // with features 4 g + q in slots q (sel0) or 4 + q (sel1) against them
  // gives lane (g, n) feature n of rows 4 g .. 4 g + 3 (the block
  // transposed, exactly).
  u32x4 sel0 = {0u, 0u, 0u, 0u}, sel1 = {0u, 0u, 0u, 0u};
  {
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
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
  f32x4 gacc[NACC];
#pragma unroll
  for (int i = 0; i < NACC; ++i) gacc[i] = zero4;
  drain_and_sync();  // weights in LDS

  auto der = [&](uint32_t half) -> float {  // DER 2
    const float v = __uint_as_float(half);
    return act == ACT_SIGMOID ? v * (1.f - v) : (act == ACT_SINE ? v : 1.f);
  };

  const int G = gridDim.x;
  for (int tile = blockIdx.x; tile < a.ntiles; tile += G) {
    const int64_t row0 = ((int64_t)tile * NW + wave) * NT * 16;  // the wave's first row
    const int64_t blk0 = row0 / 16;
    int64_t vr = M - row0;
    vr = vr < 0 ? 0 : (vr > NT * 16 ? NT * 16 : vr);
    const int vblk = (int)((vr + 15) / 16);  // valid 16-row blocks of the wave
    int64_t sb = (a.M16 - row0) / 16;
    const int sblk = (int)(sb < 0 ? 0 : (sb > NT ? NT : sb));  // blocks inside the stash

    // Activations of the wave's rows for layer l (l = 0: X), lane (g, i) of
    // block n: row 16 n + i, features 16 s + 4 g .. + 3.
    auto load_a = [&](int l, u32x2 (&ar)[NT][SW]) {
      if (l == 0) {
        const rsrc_t xr = make_rsrc(a.X + row0 * in_dim, vr * in_dim * 2);
#pragma unroll
        for (int s = 0; s < SW; ++s) {
          const int f0 = 16 * s + 4 * lg;
          if (xvec) {
            const uint32_t voff = f0 < in_dim ? (uint32_t)((li * in_dim + f0) * 2) : kOOB;
#pragma unroll
            for (int n = 0; n < NT; ++n) ar[n][s] = bload64(xr, voff, (uint32_t)(n * 32 * in_dim));
          } else {
            uint32_t vo[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) vo[r] = f0 + r < in_dim ? (uint32_t)((li * in_dim + f0 + r) * 2) : kOOB;
#pragma unroll
            for (int n = 0; n < NT; ++n) {
              uint32_t e[4];
#pragma unroll
              for (int r = 0; r < 4; ++r) e[r] = bload16(xr, vo[r], (uint32_t)(n * 32 * in_dim));
              ar[n][s] = u32x2{e[0] | (e[1] << 16), e[2] | (e[3] << 16)};
            }
          }
        }
      } else {
        const rsrc_t sr = make_rsrc(a.stashA + (size_t)(l - 1) * a.M16 * W + (size_t)row0 * W,
                                    (int64_t)sblk * 32 * W);
#pragma unroll
        for (int n = 0; n < NT; ++n)
#pragma unroll
          for (int s = 0; s < SW; ++s) ar[n][s] = bload64(sr, lane * 8, (uint32_t)((n * SW + s) * 512));
      }
    };
    // Derivative source of hidden activation idx besides A itself: the ReLU
    // mask words (DER 0) or the sine cos stash (DER 2).
    auto load_src = [&](int idx, uint32_t (&mw)[NT], u32x2 (&cs)[NT][CSW]) {
      if constexpr (DER == 0) {
        const rsrc_t mr = make_rsrc(a.reluMask + ((size_t)idx * (size_t)(a.M16 / 16) + blk0) * 64,
                                    (int64_t)vblk * 256);
#pragma unroll
        for (int n = 0; n < NT; ++n) mw[n] = bload32(mr, lane * 4, (uint32_t)(n * 256));
      } else if constexpr (DER == 2) {
        if (act == ACT_SINE) {
          const rsrc_t r = make_rsrc(a.stashS + (size_t)idx * a.M16 * W + (size_t)row0 * W,
                                     (int64_t)sblk * 32 * W);
#pragma unroll
          for (int n = 0; n < NT; ++n)
#pragma unroll
            for (int s = 0; s < SW; ++s) cs[n][s] = bload64(r, lane * 8, (uint32_t)((n * SW + s) * 512));
        }
      }
    };

    // Output delta, chain order.
    u32x4 dA[NT][KBW], dB[NT][KBW];
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) dA[n][kb] = u32x4{0u, 0u, 0u, 0u};
    {
      const rsrc_t dr = make_rsrc(a.deltaOut + row0 * OP, SEEDED ? 0 : (int64_t)vblk * 32 * OP);
      const rsrc_t cr = make_rsrc(a.cOut + row0 * OP, (SEEDED && a.cOut) ? (int64_t)vblk * 64 * OP : 0);
      const rsrc_t gr = make_rsrc(a.dY + row0 * out_dim, (SEEDED && a.dY) ? vr * out_dim * 4 : 0);
      static_for<0, OS>([&](auto sc) {
        constexpr int s = decltype(sc)::value;
        if (s >= SO) return;
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          uint32_t p0, p1;
          if constexpr (!SEEDED) {
            const u32x2 v = bload64(dr, lane * 8, (uint32_t)((n * SO + s) * 512));
            p0 = v.x;
            p1 = v.y;
          } else {
            const int64_t m = row0 + n * 16 + li;
            const int j0 = s * 16 + lg * 4;
            float g[4] = {0.f, 0.f, 0.f, 0.f};
            if (yvec) {
              const uint32_t eo = (j0 < out_dim) ? (uint32_t)(li * out_dim + j0) : kOOB / 4;
              const u32x4 v = bload128(gr, eo * 4, (uint32_t)(n * 64 * out_dim));
              g[0] = __uint_as_float(v.x);
              g[1] = __uint_as_float(v.y);
              g[2] = __uint_as_float(v.z);
              g[3] = __uint_as_float(v.w);
            } else if (m < M && j0 < out_dim) {
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
          }
          if constexpr (s & 1) {
            dA[n][s >> 1].z = p0;
            dA[n][s >> 1].w = p1;
          } else {
            dA[n][s >> 1].x = p0;
            dA[n][s >> 1].y = p1;
          }
        }
      });
    }

    u32x2 arA[NT][SW], arB[NT][SW];    // activations of layer l and l - 1
    uint32_t mwA[NT], mwB[NT];          // DER 0 mask words
    u32x2 csA[NT][CSW], csB[NT][CSW];  // DER 2 (sine) cos
#pragma unroll
    for (int n = 0; n < NT; ++n) {
      mwA[n] = mwB[n] = 0u;
#pragma unroll
      for (int s = 0; s < CSW; ++s) csA[n][s] = csB[n][s] = u32x2{0u, 0u};
    }
    load_a(L - 1, arA);
    load_src(L - 2, mwA, csA);

    // Layer l: G_l += A_l^T D_{l+1} over the wave's rows; for l >= 1 also
    // D_l = (D_{l+1} W_l^T) sigma'(a_l).  The next layer's inputs are
    // requested first, so they arrive while this layer computes.
    auto layer_step = [&](auto lc, u32x4 (&cur)[NT][KBW], u32x4 (&nxt)[NT][KBW],
                          u32x2 (&ar)[NT][SW], u32x2 (&an)[NT][SW], uint32_t (&mw)[NT],
                          uint32_t (&mn)[NT], u32x2 (&cs)[NT][CSW], u32x2 (&cn)[NT][CSW]) {
      constexpr int l = decltype(lc)::value;
      constexpr int SD = Gm::sd(l), GO = Gm::goff(l);
      if constexpr (l >= 1) load_a(l - 1, an);
      if constexpr (l >= 2) load_src(l - 2, mn, cn);
      // G_l: per 32-row step (blocks 2 k, 2 k + 1), both operands transposed
      // so that slot r holds row 4 g + r of block 2 k and slot 4 + r the same
      // row of block 2 k + 1.
#pragma unroll
      for (int k = 0; k < NT / 2; ++k) {
        u32x4 dop[SD];
#pragma unroll
        for (int j = 0; j < SD; ++j) {
          const u32x4 s0 = (j & 1) ? sel1 : sel0;
          const f32x4 o0 = mfma16(cur[2 * k][j >> 1], s0, zero4);
          const f32x4 o1 = mfma16(cur[2 * k + 1][j >> 1], s0, zero4);
          dop[j] = u32x4{pack_bf16x2(o0[0], o0[1]), pack_bf16x2(o0[2], o0[3]),
                         pack_bf16x2(o1[0], o1[1]), pack_bf16x2(o1[2], o1[3])};
        }
#pragma unroll
        for (int t = 0; t < SW; ++t) {
          const u32x4 src = {ar[2 * k][t].x, ar[2 * k][t].y, ar[2 * k + 1][t].x, ar[2 * k + 1][t].y};
          const f32x4 o0 = mfma16(src, sel0, zero4);
          const f32x4 o1 = mfma16(src, sel1, zero4);
          const u32x4 aop = {pack_bf16x2(o0[0], o0[1]), pack_bf16x2(o0[2], o0[3]),
                             pack_bf16x2(o1[0], o1[1]), pack_bf16x2(o1[2], o1[3])};
#pragma unroll
          for (int j = 0; j < SD; ++j) gacc[GO + t * SD + j] = mfma16(aop, dop[j], gacc[GO + t * SD + j]);
        }
      }
      if constexpr (l >= 1) {
        constexpr int KBL = (l == L - 1) ? KBO : KBW;
        const u32x4* wl = smem + (size_t)Gm::woff(l) * 64;
        static_for<0, SW>([&](auto sc) {
          constexpr int s = decltype(sc)::value;
          u32x4 af[KBL];
#pragma unroll
          for (int kb = 0; kb < KBL; ++kb) af[kb] = wl[(s * KBL + kb) * 64 + lane];
#pragma unroll
          for (int n = 0; n < NT; ++n) {
            f32x4 acc = zero4;
#pragma unroll
            for (int kb = 0; kb < KBL; ++kb) acc = mfma16(af[kb], cur[n][kb], acc);
            uint32_t p0, p1;
            if constexpr (DER == 0) {
              const uint32_t tm = mw[n] >> (2 * s);
              p0 = mask_halves(pack_bf16x2(acc[0], acc[1]), tm & 0x00010001u);
              p1 = mask_halves(pack_bf16x2(acc[2], acc[3]), (tm >> 1) & 0x00010001u);
            } else if constexpr (DER == 1) {
              p0 = mask_halves(pack_bf16x2(acc[0], acc[1]), nonzero_halves(ar[n][s].x));
              p1 = mask_halves(pack_bf16x2(acc[2], acc[3]), nonzero_halves(ar[n][s].y));
            } else {
              const u32x2 v = act == ACT_SINE ? cs[n][s] : ar[n][s];
              p0 = pack_bf16x2(acc[0] * der(v.x << 16), acc[1] * der(v.x & 0xffff0000u));
              p1 = pack_bf16x2(acc[2] * der(v.y << 16), acc[3] * der(v.y & 0xffff0000u));
            }
            if constexpr (s & 1) {
              nxt[n][s >> 1].z = p0;
              nxt[n][s >> 1].w = p1;
            } else {
              nxt[n][s >> 1].x = p0;
              nxt[n][s >> 1].y = p1;
            }
          }
          __builtin_amdgcn_sched_barrier(0);
        });
        if constexpr (SW == 1) {
#pragma unroll
          for (int n = 0; n < NT; ++n) {
            nxt[n][0].z = 0u;
            nxt[n][0].w = 0u;
          }
        }
      }
    };

    static_for<0, L>([&](auto ic) {
      constexpr int l = L - 1 - decltype(ic)::value;
      if constexpr (((L - 1 - l) & 1) == 0)
        layer_step(std::integral_constant<int, l>{}, dA, dB, arA, arB, mwA, mwB, csA, csB);
      else
        layer_step(std::integral_constant<int, l>{}, dB, dA, arB, arA, mwB, mwA, csB, csA);
    });
  }

  // The waves' G added in a fixed order through LDS, one layer at a time;
  // the workgroup writes one partial in the weights' layout.
  float* part = a.partial + (size_t)blockIdx.x * (size_t)a.params;
  static_for<0, L>([&](auto lc) {
    constexpr int l = decltype(lc)::value;
    constexpr int SD = Gm::sd(l), GO = Gm::goff(l);
    const int fi = l == 0 ? in_dim : W, fo = l == L - 1 ? out_dim : W;
    const int64_t off = l == 0 ? 0 : (int64_t)in_dim * W + (int64_t)(l - 1) * W * W;
    float* mine = red + (size_t)wave * W * W;
#pragma unroll
    for (int t = 0; t < SW; ++t)
#pragma unroll
      for (int j = 0; j < SD; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int k = 16 * t + 4 * lg + r, jj = 16 * j + li;
          if (k < fi && jj < fo) mine[k * fo + jj] = gacc[GO + t * SD + j][r];
        }
    __syncthreads();
    for (int e = tid; e < fi * fo; e += NW * 64) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) s += red[(size_t)w * W * W + e];
      part[off + e] = s;
    }
    __syncthreads();
  });
}

template <int W, int L, int OS, int SEEDED, int DER>
static hipError_t bwdn_launch_t(const BwdgArgs& a0, hipStream_t stream, int* grid_out) {
  using Gm = BwdnGeom<W, L, OS>;
  BwdgArgs a = a0;
  a.ntiles = (int)((a.M + kBwdnRows - 1) / kBwdnRows);
  DeviceInfo di;
  hipError_t e = device_info(&di);
  if (e != hipSuccess) return e;
  const size_t lds = Gm::lds_bytes();
  if (lds > (size_t)di.max_lds) return hipErrorNotSupported;
  auto kern = bwdn_kernel<W, L, OS, SEEDED, DER>;
  int occ = 0;
  e = kernel_occupancy(reinterpret_cast<const void*>(kern), kBwdnWaves * 64, lds, &occ);
  if (e != hipSuccess) return e;
  int grid = di.cus * occ;
  if (grid > a.ntiles) grid = a.ntiles;
  if (grid > kBwdgMaxBlocks) grid = kBwdgMaxBlocks;
  if (grid < 1) grid = 1;
  *grid_out = grid;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(kBwdnWaves * 64), lds, stream, a);
  return hipGetLastError();
}

template <int W, int OS, int DER>
static hipError_t bwdn_by_l(int L, int seeded, const BwdgArgs& a, hipStream_t s, int* g) {
  switch (L) {
    case 2: return seeded ? bwdn_launch_t<W, 2, OS, 1, DER>(a, s, g) : bwdn_launch_t<W, 2, OS, 0, DER>(a, s, g);
    case 3: return seeded ? bwdn_launch_t<W, 3, OS, 1, DER>(a, s, g) : bwdn_launch_t<W, 3, OS, 0, DER>(a, s, g);
    case 4: return seeded ? bwdn_launch_t<W, 4, OS, 1, DER>(a, s, g) : bwdn_launch_t<W, 4, OS, 0, DER>(a, s, g);
    case 5: return seeded ? bwdn_launch_t<W, 5, OS, 1, DER>(a, s, g) : bwdn_launch_t<W, 5, OS, 0, DER>(a, s, g);
    default: return hipErrorNotSupported;
  }
}

// Masks when the forward pass wrote them (DER 0), else ReLU from the stored
// activations (DER 1) or the other activations' sources (DER 2).
template <int W, int OS>
static hipError_t bwdn_by_act(int L, int seeded, const BwdgArgs& a, hipStream_t s, int* g) {
  if (a.act == ACT_RELU && a.reluMask) return bwdn_by_l<W, OS, 0>(L, seeded, a, s, g);
  if (a.act == ACT_RELU) return bwdn_by_l<W, OS, 1>(L, seeded, a, s, g);
  return bwdn_by_l<W, OS, 2>(L, seeded, a, s, g);
}

}  // namespace ffmlp
