// The whole training step of a narrow net in one kernel: the forward pass
// with the loss and the output delta, the delta loop of Algorithm 2 and the
// weight gradients G_i = A_i^T D_{i+1} (arXiv 2403.17607, section III-A;
// section V proposes fusing more of the step into one kernel).
//
// At widths 16 and 32 a wave can hold every hidden activation of its rows
// (one or two 16-feature strips per layer) and every layer's whole G (one or
// four 16x16 tiles) in VGPRs.  So each wave takes its NT 16-row blocks of a
// tile through the forward layers, keeps the activations (and for sine the
// bf16 cos of the pre-activations, the derivative source) in registers,
// computes Y, the loss and the output delta, and then runs the backward
// layers straight from those registers: the activation stash never goes to
// HBM.  Per row the kernel reads X and T (and X once more from cache for
// G_0) and writes Y only when asked.
//
// The forward arithmetic is that of the forward kernel (same k-block order,
// rounding and activation code), so Y is bitwise the same as inference; the
// backward is the per-wave scheme of the narrow fused backward (both
// contraction operands of G transposed on the matrix cores with 0/1
// selection matrices).  At the end the waves add their G and loss in a
// fixed order through LDS and each workgroup writes one partial of each
// for the fixed-order reduce kernel, so G and the loss are bitwise the same
// from run to run.
#pragma once

#include "device.h"

namespace ffmlp {

template <int W, int L, int OS>
struct TrainfGeom {
  // Two 16-row blocks per wave (one 32-row contraction step of G): at
  // width 16 four blocks took 188 VGPRs and 2 waves per SIMD, two take 128
  // and 4 (training step at 2^20 rows 43.4 -> 38.2 us).
  static constexpr int NW = kTrainfWaves, NT = 2;
  static constexpr int ROWS = NW * NT * 16;                        // rows per tile
  static constexpr int SW = W / 16, KBW = (W + 31) / 32;
  static constexpr int KBO = (OS * 16 + 31) / 32;
  // LDS fragments: the forward layers 0 .. L-1 (the output layer's OS strips
  // at most), then the backward layers 1 .. L-1.
  static constexpr int FF = (L - 1) * SW * KBW + OS * KBW;
  static constexpr int BF = (L - 1) * SW * KBW;
  static constexpr int fwd_off(int l) { return l * SW * KBW; }
  static constexpr int bwd_off(int l) { return FF + (l - 1) * SW * KBW; }
  static constexpr int sd(int l) { return l == L - 1 ? OS : SW; }  // j strips of G_l
  static constexpr int goff(int l) {
    int o = 0;
    for (int i = 0; i < l; ++i) o += SW * sd(i);
    return o;
  }
  static constexpr int nacc() { return goff(L); }
  // After the tile loop the weight LDS holds every wave's G of one layer
  // and the waves' loss sums.
  static constexpr size_t red_bytes() { return (size_t)NW * W * W * 4 + NW * 4; }
  static constexpr size_t lds_bytes() {
    return (size_t)(FF + BF) * 1024 > red_bytes() ? (size_t)(FF + BF) * 1024 : red_bytes();
  }
  static_assert((W == 16 || W == 32) && L >= 2 && L <= kTrainfMaxL && KBO == KBW,
                "fused training step: widths 16 and 32, 2 .. kTrainfMaxL matrices");
};

template <int W, int L, int OS, int ACT, bool VEC>
__global__ __launch_bounds__(kTrainfWaves * 64) void trainf_kernel(const TrainfArgs a) {
  using Gm = TrainfGeom<W, L, OS>;
  constexpr int NW = Gm::NW, NT = Gm::NT, SW = Gm::SW, KBW = Gm::KBW;
  constexpr int NACC = Gm::nacc();
  constexpr int CSL = ACT == ACT_SINE ? L - 1 : 1;  // layers of the cos source
  extern __shared__ u32x4 smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int li = lane & 15, lg = lane >> 4;
  const int64_t M = a.M;
  const int in_dim = a.in_dim, out_dim = a.out_dim, out_act = a.out_act;
  const int SO = (out_dim + 15) >> 4;
  const bool xvec = VEC || (in_dim & 7) == 0;
  const bool yvec = VEC || (out_dim & 3) == 0;

  // Resident weights, both orientations (direct-to-LDS loads).
  stage_frags(smem, a.packedF, a.fwd_total, wave, NW, lane);
  stage_frags(smem + (size_t)Gm::FF * 64, a.packedB, (uint32_t)Gm::BF, wave, NW, lane);
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
  float loss = 0.f;

  // Rows of the wave in a tile.
  struct Rows {
    int64_t row0, vr;
    int vblk;
  };
  auto rows_of = [&](int tile) {
    Rows r;
    r.row0 = ((int64_t)tile * NW + wave) * NT * 16;
    int64_t v = M - r.row0;
    r.vr = v < 0 ? 0 : (v > NT * 16 ? NT * 16 : v);
    r.vblk = (int)((r.vr + 15) / 16);
    return r;
  };

  // X of the wave's rows in input order (lane group g: features
  // 32 kb + 8 g .. + 7, the first layer's packing) and T of its output
  // strips (lane (g, i): row i, columns 16 s + 4 g .. + 3).
  u32x4 xin[NT][KBW], tq[NT][OS];
  auto load_xt = [&](int tile) {
    const Rows r = rows_of(tile);
    if (xvec) {
      const rsrc_t xr = make_rsrc(a.X + r.row0 * in_dim, r.vr * in_dim * 2);
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) {
        const int f0 = kb * 32 + lg * 8;
        const uint32_t voff = f0 < in_dim ? (uint32_t)((li * in_dim + f0) * 2) : kOOB;
#pragma unroll
        for (int n = 0; n < NT; ++n) xin[n][kb] = bload128(xr, voff, (uint32_t)(n * 32 * in_dim));
      }
    } else {
      // other input widths: one 2-byte load per feature (0 past in_dim or M)
      const rsrc_t xr = make_rsrc(a.X + r.row0 * in_dim, r.vr * in_dim * 2);
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) {
        const int f0 = kb * 32 + lg * 8;
        uint32_t vo[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) vo[q] = f0 + q < in_dim ? (uint32_t)((li * in_dim + f0 + q) * 2) : kOOB;
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          uint32_t e[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) e[q] = bload16(xr, vo[q], (uint32_t)(n * 32 * in_dim));
          xin[n][kb] = u32x4{e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16),
                             e[6] | (e[7] << 16)};
        }
      }
    }
    const rsrc_t tr = make_rsrc(a.T + r.row0 * out_dim, r.vr * out_dim * 4);
#pragma unroll
    for (int s = 0; s < OS; ++s) {
      const int j0 = s * 16 + lg * 4;
      if (yvec) {
        const uint32_t eo = (j0 < out_dim) ? (uint32_t)(li * out_dim + j0) : kOOB / 4;
#pragma unroll
        for (int n = 0; n < NT; ++n) tq[n][s] = bload128(tr, eo * 4, (uint32_t)(n * 64 * out_dim));
      } else {
        uint32_t vo[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) vo[q] = j0 + q < out_dim ? (uint32_t)((li * out_dim + j0 + q) * 4) : kOOB;
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          const uint32_t so = (uint32_t)(n * 64 * out_dim);
          tq[n][s] = u32x4{bload32(tr, vo[0], so), bload32(tr, vo[1], so), bload32(tr, vo[2], so),
                           bload32(tr, vo[3], so)};
        }
      }
    }
  };

  auto der = [&](uint32_t half) -> float {  // sigmoid a (1 - a); sine: the stored cos
    const float v = __uint_as_float(half);
    if constexpr (ACT == ACT_SIGMOID) return v * (1.f - v);
    else if constexpr (ACT == ACT_SINE) return v;
    else return 1.f;
  };

  drain_and_sync();  // weights in LDS
  const int G = gridDim.x;
  if ((int)blockIdx.x < a.ntiles) load_xt(blockIdx.x);

  for (int tile = blockIdx.x; tile < a.ntiles; tile += G) {
    const Rows r = rows_of(tile);

    // ---- forward: hidden activations a_1 .. a_{L-1} kept as strips
    // (lane (g, i) of block n: row 16 n + i, features 16 s + 4 g .. + 3).
    u32x2 st[L - 1][NT][SW];
    u32x2 cs[CSL][NT][SW];  // sine: bf16 cos of the pre-activations
    // k-block kb of layer l's input for block n, chain order
    auto in_op = [&](auto lc, int n, int kb) -> u32x4 {
      constexpr int l = decltype(lc)::value;
      if constexpr (l == 0) {
        return xin[n][kb];
      } else {
        if constexpr (SW == 1)
          return u32x4{st[l - 1][n][0].x, st[l - 1][n][0].y, 0u, 0u};
        else
          return u32x4{st[l - 1][n][2 * kb].x, st[l - 1][n][2 * kb].y, st[l - 1][n][2 * kb + 1].x,
                       st[l - 1][n][2 * kb + 1].y};
      }
    };
    static_for<0, L - 1>([&](auto lc) {
      constexpr int l = decltype(lc)::value;
      const u32x4* wl = smem + (size_t)Gm::fwd_off(l) * 64;
#pragma unroll
      for (int s = 0; s < SW; ++s) {
        u32x4 af[KBW];
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) af[kb] = wl[(s * KBW + kb) * 64 + lane];
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          f32x4 acc = zero4;
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb) acc = mfma16(af[kb], in_op(lc, n, kb), acc);
          uint32_t p0, p1;
          if constexpr (ACT == ACT_RELU) {
            p0 = relu_bf16x2(pack_bf16x2(acc[0], acc[1]));
            p1 = relu_bf16x2(pack_bf16x2(acc[2], acc[3]));
          } else {
            p0 = pack_bf16x2(act_hidden<ACT>(acc[0]), act_hidden<ACT>(acc[1]));
            p1 = pack_bf16x2(act_hidden<ACT>(acc[2]), act_hidden<ACT>(acc[3]));
          }
          st[l][n][s] = u32x2{p0, p1};
          if constexpr (ACT == ACT_SINE)
            cs[l][n][s] = u32x2{pack_bf16x2(__cosf(acc[0]), __cosf(acc[1])),
                                pack_bf16x2(__cosf(acc[2]), __cosf(acc[3]))};
        }
      }
    });

    // ---- output layer: Y, the loss and the output delta (chain order).
    u32x4 dA[NT][KBW], dB[NT][KBW];
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) dA[n][kb] = u32x4{0u, 0u, 0u, 0u};
    // One copy of the output layer per output activation (and tile class),
    // chosen once per tile.
    auto output_layer = [&](auto oc, auto fc) {
      constexpr int OA = decltype(oc)::value;
      constexpr bool FULL = decltype(fc)::value;
      const u32x4* wl = smem + (size_t)Gm::fwd_off(L - 1) * 64;
      const rsrc_t yr = make_rsrc(a.Y + r.row0 * out_dim, a.Y ? r.vr * out_dim * 2 : 0);
      static_for<0, OS>([&](auto sc) {
        constexpr int s = decltype(sc)::value;
        if (s >= SO) return;
        u32x4 af[KBW];
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) af[kb] = wl[(s * KBW + kb) * 64 + lane];
        const int j0 = s * 16 + lg * 4;
        const uint32_t eo = (j0 < out_dim) ? (uint32_t)(li * out_dim + j0) : kOOB / 4;
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          f32x4 acc = zero4;
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb)
            acc = mfma16(af[kb], in_op(std::integral_constant<int, L - 1>{}, n, kb), acc);
          bool valid[4];
          if constexpr (FULL) {
#pragma unroll
            for (int q = 0; q < 4; ++q) valid[q] = true;
          } else {
            const bool row_ok = n * 16 + li < r.vr;
#pragma unroll
            for (int q = 0; q < 4; ++q) valid[q] = row_ok && j0 + q < out_dim;
          }
          u32x2 y, d;
          train_epilogue<OA>(acc, tq[n][s], valid, a.scale, loss, y, d);
          if (a.Y != nullptr) {
            const uint32_t so = (uint32_t)(n * 32 * out_dim);
            if (yvec) {
              bstore64(y, yr, eo * 2, so);
            } else {
              // one 2-byte store per column (dropped past out_dim or M)
#pragma unroll
              for (int q = 0; q < 4; ++q)
                bstore16(((q < 2 ? y.x : y.y) >> (16 * (q & 1))) & 0xffffu, yr,
                         j0 + q < out_dim ? (uint32_t)((li * out_dim + j0 + q) * 2) : kOOB, so);
            }
          }
          if constexpr (s & 1) {
            dA[n][s >> 1].z = d.x;
            dA[n][s >> 1].w = d.y;
          } else {
            dA[n][s >> 1].x = d.x;
            dA[n][s >> 1].y = d.y;
          }
        }
      });
    };
    auto output_layer_f = [&](auto fc) {
      switch (out_act) {
        case ACT_RELU: output_layer(std::integral_constant<int, ACT_RELU>{}, fc); break;
        case ACT_SIGMOID: output_layer(std::integral_constant<int, ACT_SIGMOID>{}, fc); break;
        case ACT_SINE: output_layer(std::integral_constant<int, ACT_SINE>{}, fc); break;
        default: output_layer(std::integral_constant<int, ACT_LINEAR>{}, fc); break;
      }
    };
    // A full tile with whole output strips (the common case) needs no
    // validity masks in the epilogue (about 1% of the step at 2^20 rows).
    if (r.vr == NT * 16 && out_dim == SO * 16) output_layer_f(std::true_type{});
    else output_layer_f(std::false_type{});

    // ---- backward.  X again, as strips, for G_0 (from cache: the wave
    // read these bytes at the start of the tile); then the next tile's X
    // and T into the buffers the forward no longer needs.  That request is
    // made after the last tile too (its rows are past M and read as 0): a
    // conditional one made the wait for the strips before G_0 drain it as
    // well (width 32 at 2^20 rows 54.6 -> 53.0 us).
    u32x2 xs[NT][SW];
    {
      const rsrc_t xr = make_rsrc(a.X + r.row0 * in_dim, r.vr * in_dim * 2);
#pragma unroll
      for (int s = 0; s < SW; ++s) {
        const int f0 = 16 * s + 4 * lg;
        if (VEC || (in_dim & 3) == 0) {
          const uint32_t voff = f0 < in_dim ? (uint32_t)((li * in_dim + f0) * 2) : kOOB;
#pragma unroll
          for (int n = 0; n < NT; ++n) xs[n][s] = bload64(xr, voff, (uint32_t)(n * 32 * in_dim));
        } else {
          uint32_t vo[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) vo[q] = f0 + q < in_dim ? (uint32_t)((li * in_dim + f0 + q) * 2) : kOOB;
#pragma unroll
          for (int n = 0; n < NT; ++n) {
            uint32_t e[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) e[q] = bload16(xr, vo[q], (uint32_t)(n * 32 * in_dim));
            xs[n][s] = u32x2{e[0] | (e[1] << 16), e[2] | (e[3] << 16)};
          }
        }
      }
    }
    load_xt(tile + G);

    // Layer l: G_l += A_l^T D_{l+1} over the wave's rows; for l >= 1 also
    // D_l = (D_{l+1} W_l^T) sigma'(a_l).
    auto layer_step = [&](auto lc, const u32x4 (&cur)[NT][KBW], u32x4 (&nxt)[NT][KBW]) {
      constexpr int l = decltype(lc)::value;
      constexpr int SD = Gm::sd(l), GO = Gm::goff(l);
      const u32x2 (&ar)[NT][SW] = [&]() -> const u32x2 (&)[NT][SW] {
        if constexpr (l == 0) return xs;
        else return st[l - 1];
      }();
      // G_l, 32 rows (blocks 2 k, 2 k + 1) per step: slot q of both
      // operands holds row 4 g + q of block 2 k, slot 4 + q the same row of
      // block 2 k + 1.
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
        if constexpr (SW == 2) {
          // Width 32: each block's two strips are already one operand (the
          // forward's k-block); sel0 / sel1 transpose its strip 0 / 1.  No
          // operand is assembled from the two blocks' strips (4 register
          // moves per transpose pair).
          f32x4 o[2][2];
#pragma unroll
          for (int b = 0; b < 2; ++b) {
            const u32x4 src = {ar[2 * k + b][0].x, ar[2 * k + b][0].y, ar[2 * k + b][1].x, ar[2 * k + b][1].y};
            o[b][0] = mfma16(src, sel0, zero4);
            o[b][1] = mfma16(src, sel1, zero4);
          }
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            const u32x4 aop = {pack_bf16x2(o[0][t][0], o[0][t][1]), pack_bf16x2(o[0][t][2], o[0][t][3]),
                               pack_bf16x2(o[1][t][0], o[1][t][1]), pack_bf16x2(o[1][t][2], o[1][t][3])};
#pragma unroll
            for (int j = 0; j < SD; ++j) gacc[GO + t * SD + j] = mfma16(aop, dop[j], gacc[GO + t * SD + j]);
          }
        } else {
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
      }
      if constexpr (l >= 1) {
        const u32x4* wl = smem + (size_t)Gm::bwd_off(l) * 64;
        static_for<0, SW>([&](auto sc) {
          constexpr int s = decltype(sc)::value;
          u32x4 af[KBW];
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb) af[kb] = wl[(s * KBW + kb) * 64 + lane];
#pragma unroll
          for (int n = 0; n < NT; ++n) {
            f32x4 acc = zero4;
#pragma unroll
            for (int kb = 0; kb < KBW; ++kb) acc = mfma16(af[kb], cur[n][kb], acc);
            uint32_t p0, p1;
            if constexpr (ACT == ACT_RELU) {
              // relu'(a) = [a > 0]: zero the rounded products where a is 0
              p0 = mask_halves(pack_bf16x2(acc[0], acc[1]), nonzero_halves(ar[n][s].x));
              p1 = mask_halves(pack_bf16x2(acc[2], acc[3]), nonzero_halves(ar[n][s].y));
            } else if constexpr (ACT == ACT_LINEAR) {
              p0 = pack_bf16x2(acc[0], acc[1]);
              p1 = pack_bf16x2(acc[2], acc[3]);
            } else {
              const u32x2 v = ACT == ACT_SINE ? cs[ACT == ACT_SINE ? l - 1 : 0][n][s] : ar[n][s];
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
      if constexpr ((decltype(ic)::value & 1) == 0)
        layer_step(std::integral_constant<int, l>{}, dA, dB);
      else
        layer_step(std::integral_constant<int, l>{}, dB, dA);
    });
  }

  // The waves' G and loss added in a fixed order through LDS (the weights
  // are no longer read), one layer at a time; the workgroup writes one
  // partial of each.
  __syncthreads();
  float* red = reinterpret_cast<float*>(smem);
  float* redl = red + (size_t)NW * W * W;
  const float lw = wave_sum(loss);
  if (lane == 0) redl[wave] = lw;
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
        for (int q = 0; q < 4; ++q) {
          const int k = 16 * t + 4 * lg + q, jj = 16 * j + li;
          if (k < fi && jj < fo) mine[k * fo + jj] = gacc[GO + t * SD + j][q];
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
  if (tid == 0) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) s += redl[w];
    a.lossPart[blockIdx.x] = s;
  }
}

template <int W, int L, int OS, int ACT, bool VEC>
static hipError_t trainf_launch_t(const TrainfArgs& a0, hipStream_t stream, int* grid_out) {
  using Gm = TrainfGeom<W, L, OS>;
  TrainfArgs a = a0;
  a.ntiles = (int)((a.M + Gm::ROWS - 1) / Gm::ROWS);
  if (a.fwd_total > (uint32_t)Gm::FF) return hipErrorInvalidValue;
  DeviceInfo di;
  hipError_t e = device_info(&di);
  if (e != hipSuccess) return e;
  const size_t lds = Gm::lds_bytes();
  if (lds > (size_t)di.max_lds) return hipErrorNotSupported;
  auto kern = trainf_kernel<W, L, OS, ACT, VEC>;
  int occ = 0;
  e = kernel_occupancy(reinterpret_cast<const void*>(kern), kTrainfWaves * 64, lds, &occ);
  if (e != hipSuccess) return e;
  int grid = di.cus * occ;
  if (grid > a.ntiles) grid = a.ntiles;
  if (grid > kBwdgMaxBlocks) grid = kBwdgMaxBlocks;
  if (grid < 1) grid = 1;
  *grid_out = grid;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(kTrainfWaves * 64), lds, stream, a);
  return hipGetLastError();
}

template <int W, int OS, int ACT, bool VEC>
static hipError_t trainf_by_l(int L, const TrainfArgs& a, hipStream_t s, int* g) {
  switch (L) {
    case 2: return trainf_launch_t<W, 2, OS, ACT, VEC>(a, s, g);
    case 3: return trainf_launch_t<W, 3, OS, ACT, VEC>(a, s, g);
    case 4: return trainf_launch_t<W, 4, OS, ACT, VEC>(a, s, g);
    case 5: return trainf_launch_t<W, 5, OS, ACT, VEC>(a, s, g);
    default: return hipErrorNotSupported;
  }
}

// VEC: X rows a multiple of 8 features and Y rows of 4 (16- and 8-byte
// accesses only), the common case, compiled without the per-element paths:
// measured at 2^20 rows with the output activation also fixed, width 16
// 38.2 -> 32.5 us, width 32 63.3 -> 52.2 us, width 64 201.9 -> 182.7 us.
template <int W, int OS, int ACT>
static hipError_t trainf_by_vec(int L, const TrainfArgs& a, hipStream_t s, int* g) {
  if (a.in_dim % 8 == 0 && a.out_dim % 4 == 0) return trainf_by_l<W, OS, ACT, true>(L, a, s, g);
  return trainf_by_l<W, OS, ACT, false>(L, a, s, g);
}

template <int W, int OS>
static hipError_t trainf_by_act(int act, int L, const TrainfArgs& a, hipStream_t s, int* g) {
  switch (act) {
    case ACT_RELU: return trainf_by_vec<W, OS, ACT_RELU>(L, a, s, g);
    case ACT_SIGMOID: return trainf_by_vec<W, OS, ACT_SIGMOID>(L, a, s, g);
    case ACT_SINE: return trainf_by_vec<W, OS, ACT_SINE>(L, a, s, g);
    default: return trainf_by_vec<W, OS, ACT_LINEAR>(L, a, s, g);
  }
}

}  // namespace ffmlp
