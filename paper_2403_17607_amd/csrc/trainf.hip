// Fused training step entry: which nets it covers, and dispatch on the
// width; each width's instantiations are compiled in their own translation
// unit (trainf16.hip, trainf32.hip, trainf64.hip); the kernels are in
// trainf_kernel.h (widths 16 and 32) and trainw_kernel.h (width 64).
#include "trainf_kernel.h"

namespace ffmlp {

template <int W>
hipError_t launch_train_fused_w(int L, int act, int out_dim, const TrainfArgs& a, hipStream_t s,
                                int* grid_out);

bool train_fused_supported(int width, int L) {
  return (width == 16 || width == 32 || width == 64) && L >= 2 && L <= kTrainfMaxL;
}

hipError_t launch_train_fused(int width, int L, int act, int out_dim, const TrainfArgs& a,
                              hipStream_t s, int* grid_out) {
  if (!train_fused_supported(width, L)) return hipErrorNotSupported;
  switch (width) {
    case 16: return launch_train_fused_w<16>(L, act, out_dim, a, s, grid_out);
    case 32: return launch_train_fused_w<32>(L, act, out_dim, a, s, grid_out);
    case 64: return launch_train_fused_w<64>(L, act, out_dim, a, s, grid_out);
    default: return hipErrorNotSupported;
  }
}

}  // namespace ffmlp
