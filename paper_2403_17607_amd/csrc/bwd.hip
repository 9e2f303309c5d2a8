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
#include "device.h"

namespace ffmlp {

template <int W, int ACT, int SEEDED>
__global__ __launch_bounds__(TileCfg<W>::NW * 64) void bwd_kernel(const BwdArgs a) {
  constexpr int NT = TileCfg<W>::NT, NW = TileCfg<W>::NW, NTH = NW * 64;
  constexpr int KBW = (W + 31) / 32, SW = W / 16;
  extern __shared__ u32x4 smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int li = lane & 15, lg = lane >> 4;
  const int L = a.L, out_dim = a.out_dim, out_act = a.out_act;
  const int64_t M = a.M;
  const int SO = (out_dim + 15) >> 4;
  const int KBO = (SO + 1) >> 1;
  const bool yvec = (out_dim & 3) == 0;

  if (a.resident && L > 1) {
    copy_frags(smem, a.packed, a.total_frags, tid, NTH);
    __syncthreads();
  }
  for (int tile = blockIdx.x; tile < a.ntiles; tile += gridDim.x) {
    const int64_t tb0 = ((int64_t)tile * NW + wave) * NT;
    u32x4 d[NT][KBW];
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) d[n][kb] = u32x4{0u, 0u, 0u, 0u};

    // Output delta, in chain order.
    static_for<0, SW>([&](auto sc) {
      constexpr int s = decltype(sc)::value;
      if (s >= SO) return;
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const int64_t t16 = tb0 + n;
        uint32_t p0 = 0u, p1 = 0u;
        if (t16 * 16 < M) {
          const size_t idx = ((size_t)(t16 * SO + s) * 64 + lane) * 4;
          if constexpr (!SEEDED) {
            const u32x2 v = *reinterpret_cast<const u32x2*>(a.deltaOut + idx);
            p0 = v.x;
            p1 = v.y;
          } else {
            const int64_t m = t16 * 16 + li;
            const int j0 = s * 16 + lg * 4;
            float g[4] = {0.f, 0.f, 0.f, 0.f};
            if (m < M && j0 < out_dim) {
              const float* dr = a.dY + m * out_dim + j0;
              if (yvec) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(dr);
                g[0] = v[0]; g[1] = v[1]; g[2] = v[2]; g[3] = v[3];
              } else {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                  if (j0 + r < out_dim) g[r] = dr[r];
              }
            }
            if (out_act != ACT_LINEAR) {
              const f32x4 c = *reinterpret_cast<const f32x4*>(a.cOut + idx);
#pragma unroll
              for (int r = 0; r < 4; ++r) g[r] *= act_out_grad(out_act, c[r], act_apply(out_act, c[r]));
            }
            p0 = pack_bf16x2(g[0], g[1]);
            p1 = pack_bf16x2(g[2], g[3]);
            *reinterpret_cast<u32x2*>(a.deltaOut + idx) = u32x2{p0, p1};
          }
        }
        if (s & 1) {
          d[n][s >> 1].z = p0;
          d[n][s >> 1].w = p1;
        } else {
          d[n][s >> 1].x = p0;
          d[n][s >> 1].y = p1;
        }
      }
    });

    for (int l = L - 1; l >= 1; --l) {
      const int KB = (l == L - 1) ? KBO : KBW;
      const uint32_t off = (uint32_t)(l - 1) * a.layH_frags;
      const u32x4* wl;
      if (a.resident) {
        wl = smem + (size_t)off * 64;
      } else {
        __syncthreads();
        copy_frags(smem, a.packed + (size_t)off * 64, (uint32_t)(SW * KB), tid, NTH);
        __syncthreads();
        wl = smem;
      }
      const uint16_t* gsrc = (ACT == ACT_SINE ? a.stashS : a.stashA) + (size_t)(l - 1) * a.M16 * W;
      uint16_t* dst = a.deltaH + (size_t)(l - 1) * a.M16 * W;
      u32x4 nxt[NT][KBW];
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) nxt[n][kb] = u32x4{0u, 0u, 0u, 0u};

      static_for<0, SW>([&](auto sc) {
        constexpr int s = decltype(sc)::value;
        u32x2 gv[NT];
        if constexpr (ACT != ACT_LINEAR) {
#pragma unroll
          for (int n = 0; n < NT; ++n) {
            const int64_t t16 = tb0 + n;
            gv[n] = (t16 * 16 < M)
                        ? *reinterpret_cast<const u32x2*>(gsrc + ((size_t)(t16 * SW + s) * 64 + lane) * 4)
                        : u32x2{0u, 0u};
          }
        }
        u32x4 af[KBW];
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb)
          af[kb] = (kb < KB) ? wl[(s * KB + kb) * 64 + lane] : u32x4{0u, 0u, 0u, 0u};
        f32x4 acc[NT];
#pragma unroll
        for (int n = 0; n < NT; ++n) acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
          if (kb < KB) {
#pragma unroll
            for (int n = 0; n < NT; ++n) acc[n] = mfma16(af[kb], d[n][kb], acc[n]);
          }
        }
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          float dd[4];
          if constexpr (ACT != ACT_LINEAR) {
            dd[0] = acc[n][0] * act_hidden_grad<ACT>(bf16_lo(gv[n].x));
            dd[1] = acc[n][1] * act_hidden_grad<ACT>(bf16_hi(gv[n].x));
            dd[2] = acc[n][2] * act_hidden_grad<ACT>(bf16_lo(gv[n].y));
            dd[3] = acc[n][3] * act_hidden_grad<ACT>(bf16_hi(gv[n].y));
          } else {
            dd[0] = acc[n][0]; dd[1] = acc[n][1]; dd[2] = acc[n][2]; dd[3] = acc[n][3];
          }
          const uint32_t p0 = pack_bf16x2(dd[0], dd[1]), p1 = pack_bf16x2(dd[2], dd[3]);
          if (s & 1) {
            nxt[n][s >> 1].z = p0;
            nxt[n][s >> 1].w = p1;
          } else {
            nxt[n][s >> 1].x = p0;
            nxt[n][s >> 1].y = p1;
          }
          const int64_t t16 = tb0 + n;
          if (t16 * 16 < M)
            *reinterpret_cast<u32x2*>(dst + ((size_t)(t16 * SW + s) * 64 + lane) * 4) = u32x2{p0, p1};
        }
        // Keep each strip's work together: bounds the live registers.
        __builtin_amdgcn_sched_barrier(0);
      });
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) d[n][kb] = nxt[n][kb];
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
  a.resident = res_bytes + 1024 <= (size_t)di.max_lds ? 1 : 0;
  size_t lds = a.resident ? res_bytes : (size_t)a.layH_frags * 1024;
  if (lds == 0) lds = 16;
  auto kern = bwd_kernel<W, ACT, SEEDED>;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  int occ = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, NTH, lds);
  if (e != hipSuccess) return e;
  if (occ < 1) occ = 1;
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

hipError_t launch_backward(int width, int act, int seeded, const BwdArgs& a, hipStream_t s) {
  switch (width) {
    case 16: return by_act<16>(act, seeded, a, s);
    case 32: return by_act<32>(act, seeded, a, s);
    case 64: return by_act<64>(act, seeded, a, s);
    case 128: return by_act<128>(act, seeded, a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ffmlp
