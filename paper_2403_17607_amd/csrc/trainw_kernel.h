// The whole training step of a width-64 net in one kernel: the forward
// pass with the loss and the output delta, the delta loop of Algorithm 2
// and the weight gradients G_i = A_i^T D_{i+1} (arXiv 2403.17607, section
// III-A; section V proposes fusing more of the step into one kernel).
//
// At width 64 every layer's G (16 tiles of 16x16 per hidden layer) is too
// large for one wave, so G is split across the workgroup as in the fused
// backward kernel: wave w keeps fixed slices of every G_i in registers over
// all of its workgroup's tiles.  What that kernel reads from the stash in
// HBM, this one computes itself: a workgroup of eight waves owns a tile of
// 8 NT 16-row blocks, each wave takes its NT blocks through the forward
// layers (the forward kernel's arithmetic, so Y is bitwise the inference Y)
// and keeps every hidden activation (and for sine the bf16 cos of the
// pre-activation) in VGPRs.  NT is 2 (256-row tiles: every weight fragment
// read from LDS feeds two MFMAs) except for sine nets, whose cos source
// leaves registers for one block only.  Per backward layer each wave writes its rows' D_{i+1} and A_i,
// transposed on the matrix cores (MFMA against 0/1 selection matrices), into
// two LDS tiles DT and AT [feature][row]; after a barrier every wave
// accumulates its G slices from them over the tile's 128 rows, interleaved
// with the delta product of its own rows.  Only X, T (and Y when asked for)
// and one G and loss partial per workgroup touch HBM.
#pragma once

#include "device.h"

namespace ffmlp {

template <int L, int OS, int NT>
struct TrainwGeom {
  static constexpr int W = 64, NW = kTrainfWaves, SW = 4, KBW = 2;
  static constexpr int KBO = (OS * 16 + 31) / 32;  // k-blocks of the output delta
  static constexpr int ROWS = NW * NT * 16;        // rows per tile
  static constexpr int LDT = ROWS;                 // DT / AT row: the tile's rows in bf16
  static constexpr int KS = ROWS / 32;             // 32-row contraction steps per tile
  // LDS: forward layers 0 .. L-1 (the output layer's OS strips at most),
  // backward layers 1 .. L-2 whole and the output layer's first KBO
  // k-blocks of each strip, then DT and AT.
  static constexpr int FF = (L - 1) * SW * KBW + OS * KBW;
  static constexpr int BWF = (L - 2) * SW * KBW + SW * KBO;
  static constexpr int fwd_off(int l) { return l * SW * KBW; }
  static constexpr int bwd_off(int l) { return FF + (l - 1) * SW * KBW; }
  static constexpr size_t tiles_off() { return (size_t)(FF + BWF) * 1024; }
  static constexpr size_t lds_bytes() { return tiles_off() + (size_t)2 * W * LDT * 2; }
  // G slices: SW k-strips x sd(l) j-strips of 16x16 tiles per layer; wave w
  // owns tiles w tpw .. w tpw + tpw - 1 (row-major over (k-strip,
  // j-strip)), or tile w when there are fewer tiles than waves.
  static constexpr int sd(int l) { return l == L - 1 ? OS : SW; }
  static constexpr int ntl(int l) { return SW * sd(l); }
  static constexpr int tpw(int l) { return ntl(l) >= NW ? ntl(l) / NW : 1; }
  static constexpr int goff(int l) {
    int o = 0;
    for (int i = 0; i < l; ++i) o += tpw(i);
    return o;
  }
  static constexpr int nacc() { return goff(L); }
  static_assert(L >= 2 && L <= kTrainfMaxL && (OS == 1 || OS == 4) && (NT == 1 || NT == 2),
                "width-64 fused training step");
};

// Two blocks per wave where the registers allow it: one output strip, no
// cos source, and at most 5 matrices (3 when X or Y need the per-element
// paths).  Measured at 2^20 rows: image-like net (in 32, 2 hidden layers,
// sigmoid out 3) 110 -> 95 us, 5 matrices 181.5 -> 166 us.
template <int L, int OS, int ACT, bool VEC>
constexpr int trainw_nt() {
  return (ACT != ACT_SINE && OS == 1 && L <= (VEC ? 5 : 3)) ? 2 : 1;
}

template <int L, int OS, int ACT, bool VEC>
__global__ __launch_bounds__(kTrainfWaves * 64) void trainw_kernel(const TrainfArgs a) {
  constexpr int NT = trainw_nt<L, OS, ACT, VEC>();
  using Gm = TrainwGeom<L, OS, NT>;
  constexpr int NW = Gm::NW, SW = Gm::SW, KBW = Gm::KBW, KBO = Gm::KBO, LDT = Gm::LDT, KS = Gm::KS;
  constexpr int NACC = Gm::nacc();
  constexpr int CSL = ACT == ACT_SINE ? L - 1 : 1;  // layers of the cos source
  extern __shared__ u32x4 smem[];
  uint16_t* DT = reinterpret_cast<uint16_t*>(reinterpret_cast<uint8_t*>(smem) + Gm::tiles_off());
  uint16_t* AT = DT + (size_t)Gm::W * LDT;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int li = lane & 15, lg = lane >> 4;
  const int64_t M = a.M;
  const int in_dim = a.in_dim, out_dim = a.out_dim, out_act = a.out_act;
  const int SO = (out_dim + 15) >> 4;
  const bool xvec = VEC || (in_dim & 7) == 0;
  const bool yvec = VEC || (out_dim & 3) == 0;

  // Resident weights (direct-to-LDS loads, waited for below).
  stage_frags(smem, a.packedF, a.fwd_total, wave, NW, lane);
  stage_frags(smem + (size_t)Gm::FF * 64, a.packedB, (uint32_t)((L - 2) * SW * KBW), wave, NW, lane);
  {
    const u32x4* src = a.packedB + (size_t)(L - 2) * SW * KBW * 64;
    u32x4* dst = smem + (size_t)Gm::bwd_off(L - 1) * 64;
    for (int f = wave; f < SW * KBO; f += NW) {
      const int s = f / KBO, kb = f - s * KBO;
      __builtin_amdgcn_global_load_lds(
          (const void __attribute__((address_space(1)))*)(src + (size_t)(s * KBW + kb) * 64 + lane),
          (void __attribute__((address_space(3)))*)(dst + (size_t)f * 64), 16, 0, 0);
    }
  }
  // Selection matrices (see the fused backward kernel): an MFMA of a
  // chain-order operand (lane (g, i): row i, slots 0-3 features 4 g + q of
  // one strip, slots 4-7 of the next) against sel0 (sel1) gives lane (g, n)
  // feature n of the first (second) strip for rows 4 g .. 4 g + 3.
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

  auto slice = [&](auto lc, int& kt, int& jt0) -> bool {
    constexpr int l = decltype(lc)::value;
    constexpr int sd = Gm::sd(l), ntl = Gm::ntl(l), tpw = Gm::tpw(l);
    if constexpr (ntl >= NW) {
      const int t0 = wave * tpw;
      kt = t0 / sd;
      jt0 = t0 % sd;
      return true;
    } else {
      kt = wave / sd;
      jt0 = wave % sd;
      return wave < ntl;
    }
  };
  // Element offset of chunk c (8 rows, one 16-byte operand) of feature row f
  // in DT or AT; chunk c is stored at c ^ (f % 16) ^ 4 [f / 8 odd]: eight
  // consecutive features then use eight different bank groups, and so do
  // the features 8 (n / 4) + n % 4 that the input-order X transposes store
  // (with f % 16 alone, features f and f + 8 met there).
  auto dt_off = [&](int f, int c) { return f * LDT + ((c ^ (f & 15) ^ ((f >> 1) & 4)) << 3); };
  // Rows 4 g .. 4 g + 3 of the tile's block b (block n of wave w is
  // b = w NT + n), one feature per lane, go to chunk 4 (b / 2) + g, half
  // (b % 2) ^ (g % 2): the order in which the 16-byte reads below hand 8
  // rows to an MFMA operand, the same in both tiles, so both operands pair
  // the same rows.
  auto put_t = [&](uint16_t* tile, int f, int n, const f32x4& o) {
    const int b = wave * NT + n;
    const u32x2 v = {pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
    *reinterpret_cast<u32x2*>(tile + dt_off(f, 4 * (b >> 1) + lg) + 4 * ((b & 1) ^ (lg & 1))) = v;
  };
  // With two blocks per wave the chunk 4 w + g of feature f holds rows
  // 4 g .. 4 g + 3 of both of wave w's blocks (block 2 w in its first half),
  // written as one 16-byte store: eight lanes of one lane group then cover
  // eight different chunks, free of bank conflicts, where the 8-byte stores
  // of sixteen lanes met two to a bank (the stores took half of the
  // kernel's LDS cycles, half of them conflict stalls).
  auto put_t2 = [&](uint16_t* tile, int f, const f32x4& o0, const f32x4& o1) {
    const u32x4 v = {pack_bf16x2(o0[0], o0[1]), pack_bf16x2(o0[2], o0[3]), pack_bf16x2(o1[0], o1[1]),
                     pack_bf16x2(o1[2], o1[3])};
    *reinterpret_cast<u32x4*>(tile + dt_off(f, 4 * wave + lg)) = v;
  };

  drain_and_sync();  // weights in LDS

  struct Rows {
    int64_t row0, vr;
  };
  auto rows_of = [&](int tile) {
    Rows r;
    r.row0 = (int64_t)tile * Gm::ROWS + wave * NT * 16;
    int64_t v = M - r.row0;
    r.vr = v < 0 ? 0 : (v > NT * 16 ? NT * 16 : v);
    return r;
  };
  // X of the wave's rows in input order (lane group g of block n: features
  // 32 kb + 8 g .. + 7, the first layer's packing) and T of its output
  // strips (lane (g, i): row 16 n + i, columns 16 s + 4 g .. + 3).
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
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          uint32_t e[8];
#pragma unroll
          for (int q = 0; q < 8; ++q)
            e[q] = bload16(xr, f0 + q < in_dim ? (uint32_t)((li * in_dim + f0 + q) * 2) : kOOB,
                           (uint32_t)(n * 32 * in_dim));
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
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          uint32_t t[4];
#pragma unroll
          for (int q = 0; q < 4; ++q)
            t[q] = bload32(tr, j0 + q < out_dim ? (uint32_t)((li * out_dim + j0 + q) * 4) : kOOB,
                           (uint32_t)(n * 64 * out_dim));
          tq[n][s] = u32x4{t[0], t[1], t[2], t[3]};
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

  const int G = gridDim.x;
  if ((int)blockIdx.x < a.ntiles) load_xt(blockIdx.x);

  for (int tile = blockIdx.x; tile < a.ntiles; tile += G) {
    const Rows r = rows_of(tile);

    // ---- forward: a_1 .. a_{L-1} of the wave's rows in chain order (the
    // next layer's B operand; k-block kb holds strips 2 kb and 2 kb + 1).
    u32x4 ach[L - 1][NT][KBW];
    u32x4 cch[CSL][NT][KBW];  // sine: bf16 cos of the pre-activations, same order
    static_for<0, L - 1>([&](auto lc) {
      constexpr int l = decltype(lc)::value;
      const u32x4* wl = smem + (size_t)Gm::fwd_off(l) * 64;
      static_for<0, SW>([&](auto sc) {
        constexpr int s = decltype(sc)::value;
        u32x4 af[KBW];
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) af[kb] = wl[(s * KBW + kb) * 64 + lane];
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          f32x4 acc = zero4;
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb) {
            if constexpr (l == 0) acc = mfma16(af[kb], xin[n][kb], acc);
            else acc = mfma16(af[kb], ach[l - 1][n][kb], acc);
          }
          uint32_t p0, p1;
          if constexpr (ACT == ACT_RELU) {
            p0 = relu_bf16x2(pack_bf16x2(acc[0], acc[1]));
            p1 = relu_bf16x2(pack_bf16x2(acc[2], acc[3]));
          } else {
            p0 = pack_bf16x2(act_hidden<ACT>(acc[0]), act_hidden<ACT>(acc[1]));
            p1 = pack_bf16x2(act_hidden<ACT>(acc[2]), act_hidden<ACT>(acc[3]));
          }
          pin(p0);
          pin(p1);
          if constexpr (s & 1) {
            ach[l][n][s >> 1].z = p0;
            ach[l][n][s >> 1].w = p1;
          } else {
            ach[l][n][s >> 1].x = p0;
            ach[l][n][s >> 1].y = p1;
          }
          if constexpr (ACT == ACT_SINE) {
            const uint32_t c0 = pack_bf16x2(__cosf(acc[0]), __cosf(acc[1]));
            const uint32_t c1 = pack_bf16x2(__cosf(acc[2]), __cosf(acc[3]));
            if constexpr (s & 1) {
              cch[l][n][s >> 1].z = c0;
              cch[l][n][s >> 1].w = c1;
            } else {
              cch[l][n][s >> 1].x = c0;
              cch[l][n][s >> 1].y = c1;
            }
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      });
    });

    // ---- output layer: Y, the loss and the output delta (chain order).
    u32x4 dA[NT][KBW], dB[NT][KBW];
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) dA[n][kb] = u32x4{0u, 0u, 0u, 0u};
    // One copy of the output layer per output activation, chosen once.
    auto output_layer = [&](auto oc) {
      constexpr int OA = decltype(oc)::value;
      const u32x4* wl = smem + (size_t)Gm::fwd_off(L - 1) * 64;
      const rsrc_t yr = make_rsrc(a.Y + r.row0 * out_dim, a.Y ? r.vr * out_dim * 2 : 0);
      static_for<0, OS>([&](auto sc) {
        constexpr int s = decltype(sc)::value;
        if (s >= SO) return;
        u32x4 af[KBW];
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) af[kb] = wl[(s * KBW + kb) * 64 + lane];
        const int j0 = s * 16 + lg * 4;
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          f32x4 acc = zero4;
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb) acc = mfma16(af[kb], ach[L - 2][n][kb], acc);
          const bool row_ok = n * 16 + li < r.vr;
          bool valid[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) valid[q] = row_ok && j0 + q < out_dim;
          u32x2 y, d;
          train_epilogue<OA>(acc, tq[n][s], valid, a.scale, loss, y, d);
          if (a.Y != nullptr) {
            const uint32_t so = (uint32_t)(n * 32 * out_dim);
            if (yvec) {
              bstore64(y, yr, (j0 < out_dim) ? (uint32_t)(li * out_dim + j0) * 2 : kOOB, so);
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
    switch (out_act) {
      case ACT_RELU: output_layer(std::integral_constant<int, ACT_RELU>{}); break;
      case ACT_SIGMOID: output_layer(std::integral_constant<int, ACT_SIGMOID>{}); break;
      case ACT_SINE: output_layer(std::integral_constant<int, ACT_SINE>{}); break;
      default: output_layer(std::integral_constant<int, ACT_LINEAR>{}); break;
    }

    // ---- backward.  X of the wave's rows once more for AT (from cache: the
    // wave read these bytes at the start of the tile); then the next tile's
    // X and T into the buffers the forward no longer needs.
    u32x4 xc[NT][KBW];
    auto load_xc = [&]() {
      // input order, as for the forward (lane group g of block n: features
      // 32 kb + 8 g .. + 7): 16 or 8 contiguous bytes per lane and row
      const rsrc_t xr = make_rsrc(a.X + r.row0 * in_dim, r.vr * in_dim * 2);
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const uint32_t so = (uint32_t)(n * 32 * in_dim);
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
          const int f0 = 32 * kb + 8 * lg;
          if (xvec) {
            xc[n][kb] = bload128(xr, f0 < in_dim ? (uint32_t)((li * in_dim + f0) * 2) : kOOB, so);
          } else {
            uint32_t e[8];
#pragma unroll
            for (int q = 0; q < 8; ++q)
              e[q] = bload16(xr, f0 + q < in_dim ? (uint32_t)((li * in_dim + f0 + q) * 2) : kOOB, so);
            xc[n][kb] = u32x4{e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16),
                              e[6] | (e[7] << 16)};
          }
        }
      }
    };

    // Layer l.  Phase 1: D_{l+1} (in `cur`) and A_l (this wave's rows)
    // transposed into DT and AT.  Phase 2 (after a barrier): the wave's G_l
    // slices over the tile's rows, interleaved strip by strip with
    // D_l = (D_{l+1} W_l^T) sigma'(a_l) of its own rows into `nxt`.  A
    // barrier then frees both tiles.
    auto layer_step = [&](auto lc, const u32x4 (&cur)[NT][KBW], u32x4 (&nxt)[NT][KBW]) {
      constexpr int l = decltype(lc)::value;
      constexpr int SD = Gm::sd(l);
      // X for AT at layer 0 (from cache), then the next tile's X and T:
      // requested as the backward starts, or for 5 matrices one layer before
      // they are needed, so that they do not hold registers through the
      // deeper layers (which lets the 5-matrix net keep two blocks per wave:
      // 181.5 -> 166 us at 2^20 rows; the shorter nets are 1-2% faster with
      // the early request).  For 5 matrices the next tile's inputs go out
      // after layer 1's first barrier: requested before its transposes, a
      // register reload there waited for them (169 -> 162 us).  The next
      // tile's request is made after the last tile too (rows past M read
      // as 0), so the wait for X before layer 0 counts it instead of
      // draining it.
      if constexpr (l == (L >= 5 ? 1 : L - 1)) {
        load_xc();
        if constexpr (L < 5) load_xt(tile + G);
      }
      if constexpr (NT == 2) {
        static_for<0, SD>([&](auto sc) {
          constexpr int s = decltype(sc)::value;
          const u32x4 sl = (s & 1) ? sel1 : sel0;
          put_t2(DT, 16 * s + li, mfma16(cur[0][s >> 1], sl, zero4), mfma16(cur[1][s >> 1], sl, zero4));
        });
        static_for<0, SW>([&](auto sc) {
          constexpr int s = decltype(sc)::value;
          const u32x4 sl = (s & 1) ? sel1 : sel0;
          if constexpr (l == 0) {
            // X in input order: k-block s / 2, half s % 2 gives lane (g, n)
            // feature 32 (s / 2) + 8 (n / 4) + 4 (s % 2) + n % 4
            if (32 * (s >> 1) < in_dim)
              put_t2(AT, 32 * (s >> 1) + 8 * (li >> 2) + 4 * (s & 1) + (li & 3),
                     mfma16(xc[0][s >> 1], sl, zero4), mfma16(xc[1][s >> 1], sl, zero4));
          } else {
            put_t2(AT, 16 * s + li, mfma16(ach[l - 1][0][s >> 1], sl, zero4),
                   mfma16(ach[l - 1][1][s >> 1], sl, zero4));
          }
        });
      } else {
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          static_for<0, SD>([&](auto sc) {
            constexpr int s = decltype(sc)::value;
            put_t(DT, 16 * s + li, n, mfma16(cur[n][s >> 1], (s & 1) ? sel1 : sel0, zero4));
          });
          static_for<0, SW>([&](auto sc) {
            constexpr int s = decltype(sc)::value;
            if constexpr (l == 0) {
              if (32 * (s >> 1) < in_dim)
                put_t(AT, 32 * (s >> 1) + 8 * (li >> 2) + 4 * (s & 1) + (li & 3), n,
                      mfma16(xc[n][s >> 1], (s & 1) ? sel1 : sel0, zero4));
            } else {
              put_t(AT, 16 * s + li, n, mfma16(ach[l - 1][n][s >> 1], (s & 1) ? sel1 : sel0, zero4));
            }
          });
        }
      }
      __syncthreads();  // DT and AT hold the tile's rows
      if constexpr (L >= 5 && l == 1) load_xt(tile + G);

      int kt, jt0;
      const bool has = slice(lc, kt, jt0);
      u32x4 aop[KS];
      if (has) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          aop[ks] = *reinterpret_cast<const u32x4*>(AT + dt_off(16 * kt + li, 4 * ks + lg));
      }
      constexpr int TPW = Gm::tpw(l), GO = Gm::goff(l);
      constexpr int NG = KS * TPW;                    // G MFMAs of the slices
      constexpr int NS = l >= 1 ? SW : 1;             // interleaving steps
      constexpr int KBL = (l == L - 1) ? KBO : KBW;   // contraction over D_{l+1}'s features
      const u32x4* wl = smem + (size_t)Gm::bwd_off(l > 0 ? l : 1) * 64;
      static_for<0, NS>([&](auto sc) {
        constexpr int s = decltype(sc)::value;
        if (has) {
          static_for<s * NG / NS, (s + 1) * NG / NS>([&](auto qc) {
            constexpr int q = decltype(qc)::value;
            constexpr int ks = q / TPW, u = q % TPW;
            const u32x4 bop = *reinterpret_cast<const u32x4*>(DT + dt_off(16 * (jt0 + u) + li, 4 * ks + lg));
            gacc[GO + u] = mfma16(aop[ks], bop, gacc[GO + u]);
          });
        }
        if constexpr (l >= 1) {
          u32x4 af[KBL];
#pragma unroll
          for (int kb = 0; kb < KBL; ++kb) af[kb] = wl[(s * KBL + kb) * 64 + lane];
#pragma unroll
          for (int n = 0; n < NT; ++n) {
            f32x4 acc = zero4;
#pragma unroll
            for (int kb = 0; kb < KBL; ++kb) acc = mfma16(af[kb], cur[n][kb], acc);
            // sigma'(a_l) of strip s from this wave's own activations
            const u32x4 av = ach[l - 1][n][s >> 1];
            const u32x2 v = (s & 1) ? u32x2{av.z, av.w} : u32x2{av.x, av.y};
            uint32_t p0, p1;
            if constexpr (ACT == ACT_RELU) {
              p0 = mask_halves(pack_bf16x2(acc[0], acc[1]), nonzero_halves(v.x));
              p1 = mask_halves(pack_bf16x2(acc[2], acc[3]), nonzero_halves(v.y));
            } else if constexpr (ACT == ACT_LINEAR) {
              p0 = pack_bf16x2(acc[0], acc[1]);
              p1 = pack_bf16x2(acc[2], acc[3]);
            } else {
              u32x2 dv = v;
              if constexpr (ACT == ACT_SINE) {
                const u32x4 cv = cch[l - 1][n][s >> 1];
                dv = (s & 1) ? u32x2{cv.z, cv.w} : u32x2{cv.x, cv.y};
              }
              p0 = pack_bf16x2(acc[0] * der(dv.x << 16), acc[1] * der(dv.x & 0xffff0000u));
              p1 = pack_bf16x2(acc[2] * der(dv.y << 16), acc[3] * der(dv.y & 0xffff0000u));
            }
            if constexpr (s & 1) {
              nxt[n][s >> 1].z = p0;
              nxt[n][s >> 1].w = p1;
            } else {
              nxt[n][s >> 1].x = p0;
              nxt[n][s >> 1].y = p1;
            }
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      });
      __syncthreads();  // every wave is done reading DT and AT
    };

    static_for<0, L>([&](auto ic) {
      constexpr int l = L - 1 - decltype(ic)::value;
      if constexpr ((decltype(ic)::value & 1) == 0)
        layer_step(std::integral_constant<int, l>{}, dA, dB);
      else
        layer_step(std::integral_constant<int, l>{}, dB, dA);
    });
  }

  // The workgroup's partial G (each element in exactly one wave's slice)
  // and its loss, the waves' sums added in a fixed order through LDS.
  float* part = a.partial + (size_t)blockIdx.x * (size_t)a.params;
  static_for<0, L>([&](auto lc) {
    constexpr int l = decltype(lc)::value;
    constexpr int TPW = Gm::tpw(l), GO = Gm::goff(l);
    int kt, jt0;
    if (!slice(lc, kt, jt0)) return;
    const int fi = l == 0 ? in_dim : Gm::W, fo = l == L - 1 ? out_dim : Gm::W;
    const int64_t off = l == 0 ? 0 : (int64_t)in_dim * Gm::W + (int64_t)(l - 1) * Gm::W * Gm::W;
#pragma unroll
    for (int u = 0; u < TPW; ++u) {
      const int j = 16 * (jt0 + u) + li;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int k = 16 * kt + 4 * lg + q;
        if (k < fi && j < fo) part[off + (int64_t)k * fo + j] = gacc[GO + u][q];
      }
    }
  });
  float* redl = reinterpret_cast<float*>(DT);  // free after the tile loop's last barrier
  const float lw = wave_sum(loss);
  if (lane == 0) redl[wave] = lw;
  __syncthreads();
  if (tid == 0) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) s += redl[w];
    a.lossPart[blockIdx.x] = s;
  }
}

template <int L, int OS, int ACT, bool VEC>
static hipError_t trainw_launch_t(const TrainfArgs& a0, hipStream_t stream, int* grid_out) {
  using Gm = TrainwGeom<L, OS, trainw_nt<L, OS, ACT, VEC>()>;
  TrainfArgs a = a0;
  a.ntiles = (int)((a.M + Gm::ROWS - 1) / Gm::ROWS);
  if (a.fwd_total > (uint32_t)Gm::FF) return hipErrorInvalidValue;
  DeviceInfo di;
  hipError_t e = device_info(&di);
  if (e != hipSuccess) return e;
  const size_t lds = Gm::lds_bytes();
  if (lds > (size_t)di.max_lds) return hipErrorNotSupported;
  auto kern = trainw_kernel<L, OS, ACT, VEC>;
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

template <int OS, int ACT, bool VEC>
static hipError_t trainw_by_l(int L, const TrainfArgs& a, hipStream_t s, int* g) {
  switch (L) {
    case 2: return trainw_launch_t<2, OS, ACT, VEC>(a, s, g);
    case 3: return trainw_launch_t<3, OS, ACT, VEC>(a, s, g);
    case 4: return trainw_launch_t<4, OS, ACT, VEC>(a, s, g);
    case 5: return trainw_launch_t<5, OS, ACT, VEC>(a, s, g);
    default: return hipErrorNotSupported;
  }
}

// VEC: X rows a multiple of 8 features and Y rows of 4 (see trainf_by_vec).
template <int OS, int ACT>
static hipError_t trainw_by_vec(int L, const TrainfArgs& a, hipStream_t s, int* g) {
  if (a.in_dim % 8 == 0 && a.out_dim % 4 == 0) return trainw_by_l<OS, ACT, true>(L, a, s, g);
  return trainw_by_l<OS, ACT, false>(L, a, s, g);
}

template <int OS>
static hipError_t trainw_by_act(int act, int L, const TrainfArgs& a, hipStream_t s, int* g) {
  switch (act) {
    case ACT_RELU: return trainw_by_vec<OS, ACT_RELU>(L, a, s, g);
    case ACT_SIGMOID: return trainw_by_vec<OS, ACT_SIGMOID>(L, a, s, g);
    case ACT_SINE: return trainw_by_vec<OS, ACT_SINE>(L, a, s, g);
    default: return trainw_by_vec<OS, ACT_LINEAR>(L, a, s, g);
  }
}

}  // namespace ffmlp
