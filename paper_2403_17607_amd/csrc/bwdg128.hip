// Fused backward kernel instantiations for width 128 (the kernel is in
// bwdg_kernel.h).
#include "bwdg_kernel.h"

namespace ffmlp {

template <>
hipError_t launch_backward_fused_w<128>(int L, int out_dim, int seeded, const BwdgArgs& a,
                                        hipStream_t s, int* grid_out) {
  if (out_dim > 16) return hipErrorNotSupported;
  return bwdg_by_act<128, 1>(L, seeded, a, s, grid_out);
}

}  // namespace ffmlp
