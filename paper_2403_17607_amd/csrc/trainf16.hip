// Fused training step instantiations for width 16 (the kernel is in
// trainf_kernel.h); out_dim <= 16, so at most 1 output strip(s).
#include "trainf_kernel.h"

namespace ffmlp {

template <int W>
hipError_t launch_train_fused_w(int L, int act, int out_dim, const TrainfArgs& a, hipStream_t s,
                                int* grid_out);

template <>
hipError_t launch_train_fused_w<16>(int L, int act, int out_dim, const TrainfArgs& a, hipStream_t s,
                                    int* grid_out) {
  (void)out_dim;
  return trainf_by_act<16, 1>(act, L, a, s, grid_out);
}

}  // namespace ffmlp
