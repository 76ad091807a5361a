// down_g64.hip -- down-projection kernels for quantization groups of 64 columns.
#include "fwd_kernels.hpp"

namespace mc {
template hipError_t launch_down<2>(const Hidden&, const LayerArgs&, const mc_routing&, int,
                                    float*, size_t, int, int, hipStream_t);
}  // namespace mc
