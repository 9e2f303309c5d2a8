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
// memory).  HBM is touched for X, Y and, when training, the stash.
#include "device.h"

namespace ffmlp {

// acc[n] = (packed strip s of the layer) x act[n]: one 16-feature strip of
// C^T for the NT 16-row blocks of the wave, KB k-blocks deep.
template <int NT, int KBW>
__device__ __forceinline__ void strip_product(const u32x4* wl, int s, int KB,
                                              const u32x4 (&act)[NT][KBW], f32x4 (&acc)[NT],
                                              int lane) {
  u32x4 af[KBW];
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb)
    af[kb] = (kb < KB) ? wl[(s * KB + kb) * 64 + lane] : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
  for (int n = 0; n < NT; ++n) acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb) {
    if (kb < KB) {
#pragma unroll
      for (int n = 0; n < NT; ++n) acc[n] = mfma16(af[kb], act[n][kb], acc[n]);
    }
  }
}

template <int W, int ACT, int MODE>
__global__ __launch_bounds__(TileCfg<W>::NW * 64) void fwd_kernel(const FwdArgs a) {
  constexpr int NT = TileCfg<W>::NT, NW = TileCfg<W>::NW, NTH = NW * 64;
  constexpr int KBW = (W + 31) / 32, SW = W / 16;
  extern __shared__ u32x4 smem[];
  __shared__ float red[NW];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int li = lane & 15, lg = lane >> 4;
  const int L = a.L, in_dim = a.in_dim, out_dim = a.out_dim;
  const int64_t M = a.M;
  const int KB0 = (in_dim + 31) >> 5;
  const int SO = (out_dim + 15) >> 4;
  const bool xvec = (in_dim & 7) == 0;
  const bool yvec = (out_dim & 3) == 0;
  const int out_act = a.out_act;

  if (a.resident) {
    copy_frags(smem, a.packed, a.total_frags, tid, NTH);
    __syncthreads();
  }
  float loss = 0.f;
  for (int tile = blockIdx.x; tile < a.ntiles; tile += gridDim.x) {
    const int64_t tb0 = ((int64_t)tile * NW + wave) * NT;  // first 16-row block
    u32x4 act[NT][KBW];
    // A_1 = X in input order: lane group g takes features 32 kb + 8 g .. + 7.
#pragma unroll
    for (int n = 0; n < NT; ++n) {
      const int64_t m = (tb0 + n) * 16 + li;
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) {
        u32x4 v = {0u, 0u, 0u, 0u};
        const int f0 = kb * 32 + lg * 8;
        if (kb < KB0 && m < M && f0 < in_dim) {
          const uint16_t* xr = a.X + m * in_dim + f0;
          if (xvec) {
            v = *reinterpret_cast<const u32x4*>(xr);
          } else {
            uint32_t e[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) e[q] = (f0 + q < in_dim) ? (uint32_t)xr[q] : 0u;
            v = u32x4{e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16),
                      e[6] | (e[7] << 16)};
          }
        }
        act[n][kb] = v;
      }
    }

    // Hidden layers: A_{l+1} = bf16(sigma(A_l W_l)), kept in registers.
    for (int l = 0; l < L - 1; ++l) {
      const int KB = (l == 0) ? KB0 : KBW;
      const uint32_t off = (l == 0) ? 0u : a.lay0_frags + (uint32_t)(l - 1) * a.layH_frags;
      const u32x4* wl;
      if (a.resident) {
        wl = smem + (size_t)off * 64;
      } else {
        __syncthreads();
        copy_frags(smem, a.packed + (size_t)off * 64, (uint32_t)(SW * KB), tid, NTH);
        __syncthreads();
        wl = smem;
      }
      u32x4 nxt[NT][KBW];
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) nxt[n][kb] = u32x4{0u, 0u, 0u, 0u};

      static_for<0, SW>([&](auto sc) {
        constexpr int s = decltype(sc)::value;
        f32x4 acc[NT];
        strip_product<NT, KBW>(wl, s, KB, act, acc, lane);
        // Placed in the next layer's chain order (see common.h).
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          const uint32_t p0 = pack_bf16x2(act_hidden<ACT>(acc[n][0]), act_hidden<ACT>(acc[n][1]));
          const uint32_t p1 = pack_bf16x2(act_hidden<ACT>(acc[n][2]), act_hidden<ACT>(acc[n][3]));
          if (s & 1) {
            nxt[n][s >> 1].z = p0;
            nxt[n][s >> 1].w = p1;
          } else {
            nxt[n][s >> 1].x = p0;
            nxt[n][s >> 1].y = p1;
          }
          if constexpr (MODE != FWD_INFER) {
            const int64_t t16 = tb0 + n;
            if (t16 * 16 < M) {
              const size_t idx = (size_t)l * a.M16 * W + ((size_t)(t16 * SW + s) * 64 + lane) * 4;
              *reinterpret_cast<u32x2*>(a.stashA + idx) = u32x2{p0, p1};
              if constexpr (ACT == ACT_SINE) {
                const uint32_t c0 = pack_bf16x2(__cosf(acc[n][0]), __cosf(acc[n][1]));
                const uint32_t c1 = pack_bf16x2(__cosf(acc[n][2]), __cosf(acc[n][3]));
                *reinterpret_cast<u32x2*>(a.stashS + idx) = u32x2{c0, c1};
              }
            }
          }
        }
        // Keep each strip's work together: bounds the live registers.
        __builtin_amdgcn_sched_barrier(0);
      });
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) act[n][kb] = nxt[n][kb];
    }

    // Output layer: Y = sigma_out(C_L); when training also the loss and the
    // output delta 2 (Y - T) / (M out_dim) * sigma_out'(C_L).
    {
      const int l = L - 1;
      const int KB = (l == 0) ? KB0 : KBW;
      const uint32_t off = (l == 0) ? 0u : a.lay0_frags + (uint32_t)(l - 1) * a.layH_frags;
      const u32x4* wl;
      if (a.resident) {
        wl = smem + (size_t)off * 64;
      } else {
        __syncthreads();
        copy_frags(smem, a.packed + (size_t)off * 64, (uint32_t)(SO * KB), tid, NTH);
        __syncthreads();
        wl = smem;
      }
      for (int s = 0; s < SO; ++s) {
        f32x4 acc[NT];
        strip_product<NT, KBW>(wl, s, KB, act, acc, lane);
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          const int64_t t16 = tb0 + n;
          const int64_t m = t16 * 16 + li;
          const int j0 = s * 16 + lg * 4;
          const bool ok = (m < M) && (j0 < out_dim);
          float y[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) y[r] = act_apply(out_act, acc[n][r]);
          const uint32_t y0 = pack_bf16x2(y[0], y[1]), y1 = pack_bf16x2(y[2], y[3]);
          if (a.Y != nullptr && ok) {
            uint16_t* yr = a.Y + m * out_dim + j0;
            if (yvec) {
              *reinterpret_cast<u32x2*>(yr) = u32x2{y0, y1};
            } else {
              const uint16_t yb[4] = {(uint16_t)(y0 & 0xffff), (uint16_t)(y0 >> 16),
                                      (uint16_t)(y1 & 0xffff), (uint16_t)(y1 >> 16)};
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if (j0 + r < out_dim) yr[r] = yb[r];
            }
          }
          if constexpr (MODE == FWD_TRAIN) {
            float t[4] = {0.f, 0.f, 0.f, 0.f};
            if (ok) {
              const float* tr = a.T + m * out_dim + j0;
              if (yvec) {
                const f32x4 tv = *reinterpret_cast<const f32x4*>(tr);
                t[0] = tv[0]; t[1] = tv[1]; t[2] = tv[2]; t[3] = tv[3];
              } else {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                  if (j0 + r < out_dim) t[r] = tr[r];
              }
            }
            float d[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool valid = ok && (j0 + r < out_dim);
              const float diff = y[r] - t[r];
              if (valid) loss += diff * diff;
              d[r] = valid ? (a.scale * diff) * act_out_grad(out_act, acc[n][r], y[r]) : 0.f;
            }
            if (t16 * 16 < M) {
              const size_t idx = ((size_t)(t16 * SO + s) * 64 + lane) * 4;
              *reinterpret_cast<u32x2*>(a.deltaOut + idx) =
                  u32x2{pack_bf16x2(d[0], d[1]), pack_bf16x2(d[2], d[3])};
            }
          }
          if constexpr (MODE == FWD_STASH) {
            if (a.cOut != nullptr && t16 * 16 < M) {
              const size_t idx = ((size_t)(t16 * SO + s) * 64 + lane) * 4;
              *reinterpret_cast<f32x4*>(a.cOut + idx) = acc[n];
            }
          }
        }
      }
    }
  }

  if constexpr (MODE == FWD_TRAIN) {
    const float v = wave_sum(loss);
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

template <int W, int ACT, int MODE>
static hipError_t launch_t(const FwdArgs& a0, hipStream_t stream, int* grid_out) {
  constexpr int NTH = TileCfg<W>::NW * 64;
  FwdArgs a = a0;
  DeviceInfo di;
  hipError_t e = device_info(&di);
  if (e != hipSuccess) return e;
  const int KBW = (W + 31) / 32, SW = W / 16;
  const int KB0 = (a.in_dim + 31) / 32, SO = (a.out_dim + 15) / 16;
  uint32_t maxf = a.lay0_frags;
  if (a.L > 1) {
    maxf = maxf > (uint32_t)(SW * KBW) ? maxf : (uint32_t)(SW * KBW);
  } else {
    maxf = (uint32_t)(SO * KB0);
  }
  const size_t res_bytes = (size_t)a.total_frags * 1024;
  a.resident = res_bytes + 1024 <= (size_t)di.max_lds ? 1 : 0;
  const size_t lds = a.resident ? res_bytes : (size_t)maxf * 1024;
  auto kern = fwd_kernel<W, ACT, MODE>;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  int occ = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, NTH, lds);
  if (e != hipSuccess) return e;
  if (occ < 1) occ = 1;
  int grid = di.cus * occ;
  if (grid > a.ntiles) grid = a.ntiles;
  if (grid > kMaxLossParts) grid = kMaxLossParts;
  if (grid < 1) grid = 1;
  if (grid_out) *grid_out = grid;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(NTH), lds, stream, a);
  return hipGetLastError();
}

template <int W, int ACT>
static hipError_t by_mode(int mode, const FwdArgs& a, hipStream_t s, int* g) {
  switch (mode) {
    case FWD_INFER: return launch_t<W, ACT, FWD_INFER>(a, s, g);
    case FWD_STASH: return launch_t<W, ACT, FWD_STASH>(a, s, g);
    default: return launch_t<W, ACT, FWD_TRAIN>(a, s, g);
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

hipError_t launch_forward(int width, int act, int mode, const FwdArgs& a,
                          hipStream_t s, int* grid_out) {
  switch (width) {
    case 16: return by_act<16>(act, mode, a, s, grid_out);
    case 32: return by_act<32>(act, mode, a, s, grid_out);
    case 64: return by_act<64>(act, mode, a, s, grid_out);
    case 128: return by_act<128>(act, mode, a, s, grid_out);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ffmlp
