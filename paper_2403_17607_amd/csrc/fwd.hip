// Forward kernel entry: dispatch on the width; each width's instantiations
// are compiled in their own translation unit (fwd16.hip .. fwd128.hip), the
// kernel itself is in fwd_kernel.h.
#include "fwd_kernel.h"

namespace ffmlp {

hipError_t launch_forward(int width, int act, int mode, const FwdArgs& a,
                          hipStream_t s, int* grid_out) {
  switch (width) {
    case 16: return launch_forward_w<16>(act, mode, a, s, grid_out);
    case 32: return launch_forward_w<32>(act, mode, a, s, grid_out);
    case 64: return launch_forward_w<64>(act, mode, a, s, grid_out);
    case 128: return launch_forward_w<128>(act, mode, a, s, grid_out);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ffmlp
