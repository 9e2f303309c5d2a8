// Fused backward kernel instantiations for width 16: the per-wave variant
// (bwdn_kernel.h), which keeps every layer's whole G in each wave.
#include "bwdg_kernel.h"
#include "bwdn_kernel.h"

namespace ffmlp {

template <>
hipError_t launch_backward_fused_w<16>(int L, int out_dim, int seeded, const BwdgArgs& a,
                                        hipStream_t s, int* grid_out) {
  (void)out_dim;
  return bwdn_by_act<16, 1>(L, seeded, a, s, grid_out);
}

}  // namespace ffmlp
