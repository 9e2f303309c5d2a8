// Backward kernel instantiations for width 64 (the kernel is in bwd_kernel.h).
#include "bwd_kernel.h"

namespace ffmlp {

template <>
hipError_t launch_backward_w<64>(int act, int seeded, const BwdArgs& a, hipStream_t s) {
  return by_act<64>(act, seeded, a, s);
}

}  // namespace ffmlp
