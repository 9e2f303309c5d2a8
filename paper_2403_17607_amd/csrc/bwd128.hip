// Backward kernel instantiations for width 128 (the kernel is in bwd_kernel.h).
#include "bwd_kernel.h"

namespace ffmlp {

template <>
hipError_t launch_backward_w<128>(int act, int seeded, const BwdArgs& a, hipStream_t s) {
  return by_act<128>(act, seeded, a, s);
}

}  // namespace ffmlp
