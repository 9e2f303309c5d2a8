// Fused backward kernel instantiations for width 64 (the kernel is in
// bwdg_kernel.h).
#include "bwdg_kernel.h"

namespace ffmlp {

template <>
hipError_t launch_backward_fused_w<64>(int L, int out_dim, int seeded, const BwdgArgs& a,
                                        hipStream_t s, int* grid_out) {
  return out_dim <= 16 ? bwdg_by_act<64, 1>(L, seeded, a, s, grid_out)
                       : bwdg_by_act<64, 4>(L, seeded, a, s, grid_out);
}

}  // namespace ffmlp
