// Forward kernel instantiations for width 64 (the kernel is in fwd_kernel.h).
#include "fwd_kernel.h"

namespace ffmlp {

template <>
hipError_t launch_forward_w<64>(int act, int mode, const FwdArgs& a, hipStream_t s, int* grid_out) {
  return by_act<64>(act, mode, a, s, grid_out);
}

}  // namespace ffmlp
