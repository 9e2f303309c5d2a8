// Backward kernel entry: dispatch on the width; each width's instantiations
// are compiled in their own translation unit (bwd16.hip .. bwd128.hip), the
// kernel itself is in bwd_kernel.h.
#include "bwd_kernel.h"

namespace ffmlp {

hipError_t launch_backward(int width, int act, int seeded, const BwdArgs& a, hipStream_t s) {
  switch (width) {
    case 16: return launch_backward_w<16>(act, seeded, a, s);
    case 32: return launch_backward_w<32>(act, seeded, a, s);
    case 64: return launch_backward_w<64>(act, seeded, a, s);
    case 128: return launch_backward_w<128>(act, seeded, a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ffmlp
