// Optimizer step on fp32 master weights, then the bf16 weights the fused
// kernels read.  The paper leaves the optimizer out of its training step
// (section III-A); applications need one.  SGD, and Adam as defined by
// Kingma and Ba (2015, Algorithm 1) with bias-corrected moments; one
// thread per parameter, all state in the weights' own layout.
#include "device.h"

namespace ffmlp {

__global__ __launch_bounds__(256) void optim_kernel(const OptArgs a) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= a.n) return;
  const float g = a.G[i];
  float w = a.master[i];
  if (a.adam) {
    const float m = a.beta1 * a.m[i] + (1.f - a.beta1) * g;
    const float v = a.beta2 * a.v[i] + (1.f - a.beta2) * g * g;
    a.m[i] = m;
    a.v[i] = v;
    // lr (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
    w -= a.step_size * m / (__builtin_sqrtf(v) * a.inv_sqrt_bc2 + a.eps);
  } else {
    w -= a.lr * g;
  }
  a.master[i] = w;
  a.W[i] = __builtin_bit_cast(uint16_t, (__bf16)w);  // round to nearest even
}

hipError_t launch_optim(const OptArgs& a, hipStream_t s) {
  if (a.n == 0) return hipSuccess;
  hipLaunchKernelGGL(optim_kernel, dim3((unsigned)((a.n + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace ffmlp
