// Fused backward pass with the weight gradients: the delta loop of
// Algorithm 2, D_i = sigma_b(A_i, D_{i+1} B_i^T), and the products
// G_i = A_i^T D_{i+1} in one kernel (arXiv 2403.17607, section III-A; the
// paper computes G outside its fused kernel and names fusing it into the
// backward pass as future work in section V).
//
// The hidden activations' derivative comes from the mask words the forward
// pass wrote (DER 0: ReLU nets with masks), or, at widths up to 64, from the
// stash: [A > 0] for ReLU (DER 1) and A (1 - A) for sigmoid (DER 2) from the
// stored bf16 A (the rows of A this CU reads for its G slices anyway, so
// mostly cache hits), bf16 cos C for sine and 1 for linear (DER 2).
//
// A workgroup of eight waves owns a tile of 128 batch rows at a time
// (persistent loop over tiles).  Each wave carries the deltas of its own 16
// rows through the layers in VGPRs exactly as the unfused backward kernel
// does: chain order, backward-packed weights resident in LDS as the MFMA A
// operand, ReLU masks from the forward pass.
//
// G_i is a contraction over the batch, so its MFMA operands need each lane
// to hold batch rows of one feature, the transpose of the delta layout.
// Both operands are brought to that form on the matrix cores: an MFMA whose
// B operand is a 0/1 selection matrix returns a 16x16 block of its A operand
// transposed, exactly (one bf16 product per output, all other terms zero).
//   - Each wave writes its 16 rows of D_{i+1}, transposed, into an LDS tile
//     DT[feature][row] of the 128 rows (16-byte chunks XOR-swizzled by the
//     feature row, so that its reads and writes are free of bank conflicts).
//   - Each wave owns a fixed slice of every G_i (one 16-feature strip of A_i
//     against one or more strips of D_{i+1}).  It reads its A_i strip for
//     the tile's 128 rows straight from the activation stash, transposes it
//     the same way and accumulates the slice over the tile from DT.
// The slices stay in registers across all of the workgroup's tiles; at the
// end the workgroup writes them as one fp32 partial G, which the fixed-order
// reduce kernel adds to the other workgroups' partials.  The deltas never go
// to HBM: per row the kernel reads the output delta, the ReLU masks, X and
// the stashed activations once, and writes nothing.
#pragma once

#include "device.h"

namespace ffmlp {

template <int W, int L, int OS, bool XT8 = false>
struct BwdgGeom {
  static constexpr int NW = kBwdgWaves, SW = W / 16, KBW = (W + 31) / 32;
  static constexpr int KBO = (OS * 16 + 31) / 32;  // k-blocks of the output delta
  static constexpr int LDT = kBwdgRows;            // DT row: 128 rows of bf16, 16 chunks of 16 B
  // Resident fragments: backward layers 1 .. L-2 whole, then the output
  // layer's first KBO k-blocks of each strip (past out_dim they are zero).
  static constexpr int WFRAGS = (L - 2) * SW * KBW + SW * KBO;
  // XT, the tile's X transposed for G_0: at width 128 with 3 or more
  // matrices it takes the place of layer 1's weights (32 KiB, exactly one
  // hidden layer; LDS holds nothing else that size), which are not read
  // during layer 0 and are staged again for the next tile; otherwise it has
  // its own space after DT.
  // Only with XT8 (in_dim a multiple of 8); otherwise each wave loads its X
  // strip of the tile's rows as it loads the stash strips.
  static constexpr bool XT_REUSE = XT8 && W == 128 && L >= 3;
  static constexpr size_t xt_off() { return XT_REUSE ? 0 : (size_t)WFRAGS * 1024 + (size_t)W * LDT * 2; }
  static constexpr size_t lds_bytes() {
    return (size_t)WFRAGS * 1024 + (size_t)W * LDT * 2 + ((XT8 && !XT_REUSE) ? (size_t)W * LDT * 2 : 0);
  }
  static constexpr int woff(int l) { return (l - 1) * SW * KBW; }  // fragment offset, layer l >= 1
  // Slices of G_l: SW k-strips (features of A_l) x sd(l) j-strips (of
  // D_{l+1}) of 16x16 tiles; wave w owns tiles w tpw .. w tpw + tpw - 1
  // (row-major over (k-strip, j-strip)), or tile w when there are fewer
  // tiles than waves.
  static constexpr int sd(int l) { return l == L - 1 ? OS : SW; }
  static constexpr int ntl(int l) { return SW * sd(l); }
  static constexpr int tpw(int l) { return ntl(l) >= NW ? ntl(l) / NW : 1; }
  static constexpr int goff(int l) {
    int o = 0;
    for (int i = 0; i < l; ++i) o += tpw(i);
    return o;
  }
  static constexpr int nacc() { return goff(L); }
  static_assert(L >= 2 && L <= kBwdgMaxL, "fused backward: 2 .. kBwdgMaxL matrices");
};

// TST: stashA written transposed by the training forward (each 16-row
// block's strip s as lane (g, n) = feature 16 s + n of rows 4 g .. 4 g + 3),
// so the A operand of G_l is loaded as it is, with no transposes here.
template <int W, int L, int OS, int SEEDED, int DER, bool XT8, bool TST = false>
__global__ __launch_bounds__(kBwdgWaves * 64) void bwdg_kernel(const BwdgArgs a) {
  using Gm = BwdgGeom<W, L, OS, XT8>;
  constexpr int NW = Gm::NW, SW = Gm::SW, KBW = Gm::KBW, KBO = Gm::KBO, LDT = Gm::LDT;
  constexpr int NACC = Gm::nacc();
  constexpr int KS = kBwdgRows / 32;  // 32-row contraction steps per tile
  extern __shared__ u32x4 smem[];
  uint16_t* DT = reinterpret_cast<uint16_t*>(smem + (size_t)Gm::WFRAGS * 64);
  uint16_t* XT = reinterpret_cast<uint16_t*>(reinterpret_cast<uint8_t*>(smem) + Gm::xt_off());
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int li = lane & 15, lg = lane >> 4;
  const int64_t M = a.M;
  const int in_dim = a.in_dim, out_dim = a.out_dim, act = a.act, out_act = a.out_act;
  const bool xvec = (in_dim & 3) == 0;
  const int SO = (out_dim + 15) >> 4;  // strips of the output (at most OS)
  const int OP = SO * 16;
  const bool yvec = (out_dim & 3) == 0;

  // Resident weights (direct-to-LDS loads, waited for below).
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
  // Selection matrices (MFMA B operands, lane (g, n) holds rows 8 g .. 8 g + 7
  // of column n): sel0 picks contraction slot n - 4 g of group g, i.e. the
  // four features a lane group holds in slots 0-3; sel1 the same in slots
  // 4-7.  An A operand whose lane (g, i) holds batch row i with features
  // 4 g + q in slots q (sel0) or 4 + q (sel1) then yields out[i][n] = that
  // row's feature n, and the result lane (g, n) holds feature n of rows
  // 4 g .. 4 g + 3: the 16x16 block transposed.
  u32x4 sel0 = {0u, 0u, 0u, 0u}, sel1 = {0u, 0u, 0u, 0u};
  {
    const int q = li - 4 * lg;
    if (q >= 0 && q < 4) {
      const uint32_t one = 0x3F80u << (16 * (q & 1));  // bf16 1.0 in the slot's half
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

  // The wave's slice of G_l: its k-strip and first j-strip; false when the
  // layer has fewer tiles than waves and this wave has none.
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

  // DT element offset of chunk c (8 bf16, one 16-byte contraction operand)
  // of feature row f.  A row is 256 bytes, all 64 banks; chunk c is stored
  // at chunk c ^ (f % 16), so the 16 lanes of a 16-byte read (16 feature
  // rows, one chunk) and the 32 lanes of an 8-byte write (16 rows, two
  // chunks, different halves where they meet) touch distinct banks.
  auto dt_off = [&](int f, int c) { return f * LDT + ((c ^ (f & 15)) << 3); };

  drain_and_sync();  // weights in LDS

  // Rows of a tile: tr0 is its first row; this wave owns 16-row block `blk`
  // (valid when vblk); tvblk of the tile's blocks lie inside the stash.
  struct TileGeom {
    int64_t tr0, row0, blk, vrows;
    int vblk, tvblk;
  };
  auto geom = [&](int tile) {
    TileGeom t;
    t.tr0 = (int64_t)tile * kBwdgRows;
    t.row0 = t.tr0 + wave * 16;
    t.blk = t.row0 / 16;
    int64_t v = M - t.row0;
    t.vrows = v < 0 ? 0 : (v > 16 ? 16 : v);
    t.vblk = t.vrows > 0 ? 1 : 0;
    const int64_t tb = (a.M16 - t.tr0) / 16;
    t.tvblk = (int)(tb < 0 ? 0 : (tb > NW ? NW : tb));
    return t;
  };

  // A_l strip of the wave's G_l slice, rows tr0 .. tr0 + 127, lane (g, i)
  // of block b holding row 16 b + i, features 16 kt + 4 g .. + 3 (l >= 1,
  // from the stash).  For l = 0 with XT8 (in_dim a multiple of 8) instead
  // the wave's own 16 rows of X, every feature, in input order (lane group
  // g: features 32 kb + 8 g .. + 7 in ar[2 kb], ar[2 kb + 1]): whole rows are
  // contiguous in X, so these loads use every byte of the lines they touch,
  // where a 16-feature strip of 128 rows uses a quarter of each (measured:
  // 38 us of the 2^20-row training step at width 128); the waves transpose
  // them into XT for G_0.  Other input widths load the X strip.
  u32x2 ar[NW];
  auto load_a = [&](auto lc, const TileGeom& t) {
    constexpr int l = decltype(lc)::value;
    if constexpr (l == 0 && XT8) {
      static_assert(2 * KBW <= NW, "a wave's X rows fit the strip registers");
      const rsrc_t xr = make_rsrc(a.X + t.row0 * in_dim, t.vrows * in_dim * 2);
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) {
        const int f0 = 32 * kb + 8 * lg;
        const u32x4 v = bload128(xr, f0 < in_dim ? (uint32_t)((li * in_dim + f0) * 2) : kOOB, 0u);
        ar[2 * kb] = u32x2{v.x, v.y};
        ar[2 * kb + 1] = u32x2{v.z, v.w};
      }
    } else if constexpr (l == 0) {
      int kt, jt0;
      if (!slice(lc, kt, jt0)) return;
      int64_t rows = M - t.tr0;
      rows = rows < 0 ? 0 : (rows > kBwdgRows ? kBwdgRows : rows);
      const rsrc_t xr = make_rsrc(a.X + t.tr0 * in_dim, rows * in_dim * 2);
      const int f0 = 16 * kt + 4 * lg;
      if (xvec) {
        // in_dim a multiple of 4: the lane's four features in one 8-byte load
        const uint32_t voff = f0 < in_dim ? (uint32_t)((li * in_dim + f0) * 2) : kOOB;
#pragma unroll
        for (int b = 0; b < NW; ++b) ar[b] = bload64(xr, voff, (uint32_t)(b * 32 * in_dim));
      } else {
        // other input widths: one 2-byte load per feature (zero past in_dim)
        uint32_t vo[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) vo[r] = f0 + r < in_dim ? (uint32_t)((li * in_dim + f0 + r) * 2) : kOOB;
#pragma unroll
        for (int b = 0; b < NW; ++b) {
          uint32_t e[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) e[r] = bload16(xr, vo[r], (uint32_t)(b * 32 * in_dim));
          ar[b] = u32x2{e[0] | (e[1] << 16), e[2] | (e[3] << 16)};
        }
      }
    } else {
      int kt, jt0;
      if (!slice(lc, kt, jt0)) return;
      const rsrc_t sr = make_rsrc(a.stashA + (size_t)(l - 1) * a.M16 * W + (size_t)t.tr0 * W,
                                  (int64_t)t.tvblk * 32 * W);
      if constexpr (TST) {
        // block pair (2 ks, 2 ks + 1) into ar[2 ks], ar[2 ks + 1] in the
        // order of the operand below: odd lane groups take block 2 ks + 1
        // first (the per-lane offset picks the block; no register moves)
        const uint32_t sw = (uint32_t)(lg & 1) * SW * 512;
#pragma unroll
        for (int ks = 0; ks < NW / 2; ++ks) {
          const uint32_t so = (uint32_t)((2 * ks * SW + kt) * 512);
          ar[2 * ks] = bload64(sr, lane * 8 + sw, so);
          ar[2 * ks + 1] = bload64(sr, lane * 8 + (SW * 512 - sw), so);
        }
      } else {
#pragma unroll
        for (int b = 0; b < NW; ++b) ar[b] = bload64(sr, lane * 8, (uint32_t)((b * SW + kt) * 512));
      }
    }
  };
  auto load_mask = [&](int idx, const TileGeom& t) -> uint32_t {
    const rsrc_t mr = make_rsrc(a.reluMask + ((size_t)idx * (size_t)(a.M16 / 16) + t.blk) * 64,
                                t.vblk ? 256 : 0);
    return bload32(mr, lane * 4, 0u);
  };
  // DER = 1: the derivative source of hidden activation idx (stash index),
  // the wave's own 16 rows, all strips (none for linear layers).
  auto load_der = [&](int idx, const TileGeom& t, u32x2 (&sv)[SW]) {
    if (act == ACT_LINEAR) return;
    const uint16_t* src = act == ACT_SINE ? a.stashS : a.stashA;
    const rsrc_t r = make_rsrc(src + (size_t)idx * a.M16 * W + (size_t)t.row0 * W,
                               (int64_t)t.vblk * 32 * W);
#pragma unroll
    for (int s = 0; s < SW; ++s) sv[s] = bload64(r, lane * 8, (uint32_t)(s * 512));
  };
  // The derivative of the hidden activation from its source value (DER 2):
  // sigmoid a (1 - a) of the stored bf16 a, sine the stored bf16 cos c,
  // linear 1.
  auto der = [&](uint32_t half) -> float {
    const float v = __uint_as_float(half);
    return act == ACT_SIGMOID ? v * (1.f - v) : (act == ACT_SINE ? v : 1.f);
  };
  // What a tile needs first, requested one tile ahead (during the previous
  // tile's last layer): the output delta (training mode), the mask words of
  // a_{L-1} and the A strip of layer L-1.
  u32x2 dq[OS];
  uint32_t mq = 0u;
  u32x2 svq[DER ? SW : 1], sv[DER ? SW : 1];  // derivative sources (DER 1, 2)
#pragma unroll
  for (int s = 0; s < (DER ? SW : 1); ++s) svq[s] = sv[s] = u32x2{0u, 0u};
  auto fetch = [&](int tile) {
    const TileGeom t = geom(tile);
    if constexpr (!SEEDED) {
      const rsrc_t dr = make_rsrc(a.deltaOut + t.row0 * OP, (int64_t)t.vblk * 32 * OP);
#pragma unroll
      for (int s = 0; s < OS; ++s)
        dq[s] = bload64(dr, lane * 8, s < SO ? (uint32_t)(s * 512) : kOOB);
    }
    if constexpr (DER == 0) mq = load_mask(L - 2, t);
    else load_der(L - 2, t, svq);
    load_a(std::integral_constant<int, L - 1>{}, t);
  };

  const int G = gridDim.x;
  if ((int)blockIdx.x < a.ntiles) fetch(blockIdx.x);
  for (int tile = blockIdx.x; tile < a.ntiles; tile += G) {
    const TileGeom t = geom(tile);
    const bool more = tile + G < a.ntiles;

    // Output delta of the wave's rows, chain order.
    u32x4 dA[KBW], dB[KBW];
#pragma unroll
    for (int kb = 0; kb < KBW; ++kb) dA[kb] = u32x4{0u, 0u, 0u, 0u};
    {
      const rsrc_t cr = make_rsrc(a.cOut + t.row0 * OP, (SEEDED && a.cOut) ? (int64_t)t.vblk * 64 * OP : 0);
      const rsrc_t gr = make_rsrc(a.dY + t.row0 * out_dim, (SEEDED && a.dY) ? t.vrows * out_dim * 4 : 0);
      static_for<0, OS>([&](auto sc) {
        constexpr int s = decltype(sc)::value;
        uint32_t p0, p1;
        if constexpr (!SEEDED) {
          p0 = dq[s].x;
          p1 = dq[s].y;
        } else {
          if (s >= SO) return;
          const int64_t m = t.row0 + li;
          const int j0 = s * 16 + lg * 4;
          float g[4] = {0.f, 0.f, 0.f, 0.f};
          if (yvec) {
            const uint32_t eo = (j0 < out_dim) ? (uint32_t)(li * out_dim + j0) : kOOB / 4;
            const u32x4 v = bload128(gr, eo * 4, 0u);
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
            const u32x4 cv = bload128(cr, lane * 16, (uint32_t)(s * 1024));
            const float c[4] = {__uint_as_float(cv.x), __uint_as_float(cv.y),
                                __uint_as_float(cv.z), __uint_as_float(cv.w)};
#pragma unroll
            for (int r = 0; r < 4; ++r) g[r] *= act_out_grad(out_act, c[r], act_apply(out_act, c[r]));
          }
          p0 = pack_bf16x2(g[0], g[1]);
          p1 = pack_bf16x2(g[2], g[3]);
        }
        if constexpr (s & 1) {
          dA[s >> 1].z = p0;
          dA[s >> 1].w = p1;
        } else {
          dA[s >> 1].x = p0;
          dA[s >> 1].y = p1;
        }
      });
    }
    uint32_t mw = mq;  // relu'(a_{L-1})
    if constexpr (DER != 0) {
#pragma unroll
      for (int s = 0; s < SW; ++s) sv[s] = svq[s];
    }

    // Layer l.  Phase 1: D_{l+1} (in `cur`) transposed into DT.  Phase 2
    // (after a barrier): the wave's slice of G_l = A_l^T D_{l+1} over the
    // tile, interleaved strip by strip with D_l = (D_{l+1} W_l^T) relu'(a_l)
    // into `nxt` (independent work for the matrix cores while DT reads and
    // weight reads are in flight).  A barrier then frees DT.
    auto layer_step = [&](auto lc, u32x4 (&cur)[KBW], u32x4 (&nxt)[KBW]) {
      constexpr int l = decltype(lc)::value;
      constexpr int SD = Gm::sd(l);
      static_for<0, SD>([&](auto sc) {
        constexpr int s = decltype(sc)::value;
        const f32x4 o = mfma16(cur[s >> 1], (s & 1) ? sel1 : sel0, zero4);
        const u32x2 v = {pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
        // rows 4 g .. 4 g + 3 of block `wave` go to chunk 4 (wave / 2) + g
        // of feature row 16 s + n, half (wave % 2) ^ (g % 2): the order of
        // the transposed A operand below
        *reinterpret_cast<u32x2*>(DT + dt_off(16 * s + li, 4 * (wave >> 1) + lg) +
                                  4 * ((wave & 1) ^ (lg & 1))) = v;
      });
      if constexpr (l == 0 && XT8) {
        // XT: this wave's rows of X transposed, in DT's layout.  The k-block
        // kb operand holds features 32 kb + 8 g + q (q < 8) in lane group g,
        // so sel0 (sel1) gives lane (g, n) feature 32 kb + 8 (n / 4) + n % 4
        // (+ 4) of rows 4 g .. 4 g + 3.
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
          const u32x4 src = {ar[2 * kb].x, ar[2 * kb].y, ar[2 * kb + 1].x, ar[2 * kb + 1].y};
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const f32x4 o = mfma16(src, h ? sel1 : sel0, zero4);
            const int f = 32 * kb + 8 * (li >> 2) + 4 * h + (li & 3);
            *reinterpret_cast<u32x2*>(XT + dt_off(f, 4 * (wave >> 1) + lg) + 4 * ((wave & 1) ^ (lg & 1))) =
                u32x2{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
          }
        }
      }
      // DT (and at layer 0 XT) hold all 128 rows.  Before layer 1 the wave
      // also waits for its share of layer 1's weights, staged again after
      // the previous tile's layer 0 when XT used their space.
      if constexpr (Gm::XT_REUSE && l == 1) drain_and_sync();
      else __syncthreads();

      int kt, jt0;
      const bool has = slice(lc, kt, jt0);
      // A_l strip transposed: step ks holds rows 4 g + r of blocks 2 ks
      // (slots r) and 2 ks + 1 (slots 4 + r), feature 16 kt + n in lane
      // (g, n), the order the DT writes above used (odd lane groups hold
      // block 2 ks + 1 in slots 0-3, see dt_off)
      u32x4 aop[KS];
      if (XT8 && has && l == 0) {
        // X strip kt of the tile's rows from XT, in DT's row order
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          aop[ks] = *reinterpret_cast<const u32x4*>(XT + dt_off(16 * kt + li, 4 * ks + lg));
      } else if (TST && l >= 1 && has) {  // X for G_0 keeps the transposes
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) aop[ks] = u32x4{ar[2 * ks].x, ar[2 * ks].y, ar[2 * ks + 1].x, ar[2 * ks + 1].y};
      } else if (has) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const u32x4 src = {ar[2 * ks].x, ar[2 * ks].y, ar[2 * ks + 1].x, ar[2 * ks + 1].y};
          const f32x4 o0 = mfma16(src, sel0, zero4);
          const f32x4 o1 = mfma16(src, sel1, zero4);
          const uint32_t b00 = pack_bf16x2(o0[0], o0[1]), b01 = pack_bf16x2(o0[2], o0[3]);
          const uint32_t b10 = pack_bf16x2(o1[0], o1[1]), b11 = pack_bf16x2(o1[2], o1[3]);
          aop[ks] = (lg & 1) ? u32x4{b10, b11, b00, b01} : u32x4{b00, b01, b10, b11};
        }
      }
      // ar is free: the next layer's strip, or the next tile's first inputs
      if constexpr (l >= 1) {
        load_a(std::integral_constant<int, l - 1>{}, t);
      } else {
        if (more) fetch(tile + G);
      }
      constexpr int TPW = Gm::tpw(l), GO = Gm::goff(l);
      constexpr int NG = KS * TPW;              // G MFMAs of the slice
      constexpr int NS = l >= 1 ? SW : 1;       // interleaving steps
      constexpr int KBL = (l == L - 1) ? KBO : KBW;  // contraction over D_{l+1}'s features
      const u32x4* wl = smem + (size_t)Gm::woff(l > 0 ? l : 1) * 64;
      if constexpr (l >= 1 && SW == 1) {
        nxt[0].z = 0u;
        nxt[0].w = 0u;
      }
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
          f32x4 acc = zero4;
#pragma unroll
          for (int kb = 0; kb < KBL; ++kb) acc = mfma16(af[kb], cur[kb], acc);
          uint32_t p0, p1;
          if constexpr (DER == 0) {
            // relu'(a) is [a > 0]: zero the rounded products where a is 0
            const uint32_t tm = mw >> (2 * s);
            p0 = mask_halves(pack_bf16x2(acc[0], acc[1]), tm & 0x00010001u);
            p1 = mask_halves(pack_bf16x2(acc[2], acc[3]), (tm >> 1) & 0x00010001u);
          } else if constexpr (DER == 1) {
            // ReLU from the stored activations: each bf16 half of a is >= 0,
            // so its 0/1 multiplier is min(a, 1) as an unsigned 16-bit value
            p0 = mask_halves(pack_bf16x2(acc[0], acc[1]), nonzero_halves(sv[s].x));
            p1 = mask_halves(pack_bf16x2(acc[2], acc[3]), nonzero_halves(sv[s].y));
          } else {
            p0 = pack_bf16x2(acc[0] * der(sv[s].x << 16), acc[1] * der(sv[s].x & 0xffff0000u));
            p1 = pack_bf16x2(acc[2] * der(sv[s].y << 16), acc[3] * der(sv[s].y & 0xffff0000u));
          }
          if constexpr (s & 1) {
            nxt[s >> 1].z = p0;
            nxt[s >> 1].w = p1;
          } else {
            nxt[s >> 1].x = p0;
            nxt[s >> 1].y = p1;
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      });
      if constexpr (l >= 2) {
        if constexpr (DER == 0) mw = load_mask(l - 2, t);
        else load_der(l - 2, t, sv);
      }
      __syncthreads();  // every wave is done reading DT (and XT)
      if constexpr (Gm::XT_REUSE && l == 0) {
        // XT's space back to layer 1's weights for the next tile (waited
        // for before that tile's layer 1)
        if (more) stage_frags(smem + (size_t)Gm::woff(1) * 64, a.packed, (uint32_t)(SW * KBW), wave, NW, lane);
      }
    };

    static_for<0, L>([&](auto ic) {
      constexpr int l = L - 1 - decltype(ic)::value;
      if constexpr (((L - 1 - l) & 1) == 0)
        layer_step(std::integral_constant<int, l>{}, dA, dB);
      else
        layer_step(std::integral_constant<int, l>{}, dB, dA);
    });
  }

  // The workgroup's partial G, in the weights' layout (each element of G is
  // in exactly one wave's slice).
  float* part = a.partial + (size_t)blockIdx.x * (size_t)a.params;
  static_for<0, L>([&](auto lc) {
    constexpr int l = decltype(lc)::value;
    constexpr int TPW = Gm::tpw(l), GO = Gm::goff(l);
    int kt, jt0;
    if (!slice(lc, kt, jt0)) return;
    const int fi = l == 0 ? in_dim : W, fo = l == L - 1 ? out_dim : W;
    const int64_t off = l == 0 ? 0 : (int64_t)in_dim * W + (int64_t)(l - 1) * W * W;
#pragma unroll
    for (int u = 0; u < TPW; ++u) {
      const int j = 16 * (jt0 + u) + li;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int k = 16 * kt + 4 * lg + r;
        if (k < fi && j < fo) part[off + (int64_t)k * fo + j] = gacc[GO + u][r];
      }
    }
  });
}

template <int W, int L, int OS, int SEEDED, int DER, bool XT8, bool TST = false>
static hipError_t bwdg_launch_t1(const BwdgArgs& a, hipStream_t stream, int* grid_out) {
  using Gm = BwdgGeom<W, L, OS, XT8>;
  DeviceInfo di;
  hipError_t e = device_info(&di);
  if (e != hipSuccess) return e;
  const size_t lds = Gm::lds_bytes();
  if (lds > (size_t)di.max_lds) return hipErrorNotSupported;
  auto kern = bwdg_kernel<W, L, OS, SEEDED, DER, XT8, TST>;
  int occ = 0;
  e = kernel_occupancy(reinterpret_cast<const void*>(kern), kBwdgWaves * 64, lds, &occ);
  if (e != hipSuccess) return e;
  int grid = di.cus * occ;
  if (grid > a.ntiles) grid = a.ntiles;
  if (grid > kBwdgMaxBlocks) grid = kBwdgMaxBlocks;
  if (grid < 1) grid = 1;
  *grid_out = grid;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(kBwdgWaves * 64), lds, stream, a);
  return hipGetLastError();
}

// XT8: the X tile exchanged through LDS for G_0 (in_dim a multiple of 8).
template <int W, int L, int OS, int SEEDED, int DER>
static hipError_t bwdg_launch_t(const BwdgArgs& a, hipStream_t stream, int* grid_out) {
  if (a.stash_t) {
    // the transposed stash exists only for the training step at width 128
    if constexpr (W == 128 && SEEDED == 0 && DER == 0) {
      if (a.in_dim % 8 == 0) return bwdg_launch_t1<W, L, OS, SEEDED, DER, true, true>(a, stream, grid_out);
      return bwdg_launch_t1<W, L, OS, SEEDED, DER, false, true>(a, stream, grid_out);
    }
    return hipErrorInvalidValue;
  }
  if (a.in_dim % 8 == 0) return bwdg_launch_t1<W, L, OS, SEEDED, DER, true>(a, stream, grid_out);
  return bwdg_launch_t1<W, L, OS, SEEDED, DER, false>(a, stream, grid_out);
}

template <int W, int OS, int DER>
static hipError_t bwdg_by_l(int L, int seeded, const BwdgArgs& a, hipStream_t s, int* g) {
  switch (L) {
    case 2: return seeded ? bwdg_launch_t<W, 2, OS, 1, DER>(a, s, g) : bwdg_launch_t<W, 2, OS, 0, DER>(a, s, g);
    case 3: return seeded ? bwdg_launch_t<W, 3, OS, 1, DER>(a, s, g) : bwdg_launch_t<W, 3, OS, 0, DER>(a, s, g);
    case 4: return seeded ? bwdg_launch_t<W, 4, OS, 1, DER>(a, s, g) : bwdg_launch_t<W, 4, OS, 0, DER>(a, s, g);
    case 5: return seeded ? bwdg_launch_t<W, 5, OS, 1, DER>(a, s, g) : bwdg_launch_t<W, 5, OS, 0, DER>(a, s, g);
    default: return hipErrorNotSupported;
  }
}
// ReLU nets with mask words read them (DER 0); widths up to 64 also take
// the derivative from the stash (DER 1 for ReLU, 2 for the others).
template <int W, int OS>
static hipError_t bwdg_by_act(int L, int seeded, const BwdgArgs& a, hipStream_t s, int* g) {
  if (a.act == ACT_RELU && a.reluMask) return bwdg_by_l<W, OS, 0>(L, seeded, a, s, g);
  if constexpr (W <= 64) {
    if (a.act == ACT_RELU) return bwdg_by_l<W, OS, 1>(L, seeded, a, s, g);
    return bwdg_by_l<W, OS, 2>(L, seeded, a, s, g);
  }
  return hipErrorNotSupported;
}

template <int W>
hipError_t launch_backward_fused_w(int L, int out_dim, int seeded, const BwdgArgs& a, hipStream_t s,
                                   int* grid_out);

}  // namespace ffmlp
