// decode_g128.hip -- decode GEMVs (gate/up and down) for quantization groups of 128 columns.
#include "decode.hpp"

namespace mc {
template hipError_t launch_decode<1, true>(const LayerArgs&, const DecodeArgs&, hipStream_t);
template hipError_t launch_decode<1, false>(const LayerArgs&, const DecodeArgs&, hipStream_t);
}  // namespace mc
