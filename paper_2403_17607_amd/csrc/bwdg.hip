// Fused backward kernel entry: which nets it covers, and dispatch on the
// width; each width's instantiations are compiled in their own translation
// unit (bwdg16.hip .. bwdg128.hip), the kernel itself is in bwdg_kernel.h.
#include "bwdg_kernel.h"

namespace ffmlp {

bool backward_fused_supported(int width, int L, int act, int in_dim, int out_dim) {
  (void)in_dim;
  if (L < 2 || L > kBwdgMaxL) return false;
  if (width == 128) return act == ACT_RELU && out_dim <= 16;  // register budget
  return width == 16 || width == 32 || width == 64;
}

hipError_t launch_backward_fused(int width, int L, int out_dim, int seeded, const BwdgArgs& a,
                                 hipStream_t s, int* grid_out) {
  switch (width) {
    case 16: return launch_backward_fused_w<16>(L, out_dim, seeded, a, s, grid_out);
    case 32: return launch_backward_fused_w<32>(L, out_dim, seeded, a, s, grid_out);
    case 64: return launch_backward_fused_w<64>(L, out_dim, seeded, a, s, grid_out);
    case 128: return launch_backward_fused_w<128>(L, out_dim, seeded, a, s, grid_out);
    default: return hipErrorNotSupported;
  }
}

}  // namespace ffmlp
