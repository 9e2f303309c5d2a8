// Fused training step instantiations for width 64 (the kernel is in
// trainw_kernel.h): one output strip (out_dim <= 16) or four.
#include "trainw_kernel.h"

namespace ffmlp {

template <int W>
hipError_t launch_train_fused_w(int L, int act, int out_dim, const TrainfArgs& a, hipStream_t s,
                                int* grid_out);

template <>
hipError_t launch_train_fused_w<64>(int L, int act, int out_dim, const TrainfArgs& a, hipStream_t s,
                                    int* grid_out) {
  return out_dim <= 16 ? trainw_by_act<1>(act, L, a, s, grid_out) : trainw_by_act<4>(act, L, a, s, grid_out);
}

}  // namespace ffmlp
