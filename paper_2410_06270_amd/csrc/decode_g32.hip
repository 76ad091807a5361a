// decode_g32.hip -- decode GEMVs (gate/up and down) for quantization groups of 32 columns.
#include "decode.hpp"

namespace mc {
template hipError_t launch_decode<4, true>(const LayerArgs&, const DecodeArgs&, hipStream_t);
template hipError_t launch_decode<4, false>(const LayerArgs&, const DecodeArgs&, hipStream_t);
}  // namespace mc
