// gateup_g32.hip -- gate/up kernels for quantization groups of 32 columns.
#include "fwd_kernels.hpp"

namespace mc {
template hipError_t launch_gateup<4>(const uint16_t*, const LayerArgs&, const mc_routing&,
                                      const Hidden&, int, int, hipStream_t);
}  // namespace mc
