// gateup_g128.hip -- gate/up kernels for quantization groups of 128 columns.
#include "fwd_kernels.hpp"

namespace mc {
template hipError_t launch_gateup<1>(const uint16_t*, const LayerArgs&, const mc_routing&,
                                      const Hidden&, int, int, hipStream_t);
}  // namespace mc
