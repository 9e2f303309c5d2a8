// Forward kernel instantiations for width 128 (the kernel is in fwd_kernel.h).
#include "fwd_kernel.h"

namespace ffmlp {

template <>
hipError_t launch_forward_w<128>(int act, int mode, const FwdArgs& a, hipStream_t s, int* grid_out) {
  return by_act<128>(act, mode, a, s, grid_out);
}

}  // namespace ffmlp
