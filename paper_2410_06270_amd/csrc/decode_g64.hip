// decode_g64.hip -- decode GEMVs (gate/up and down) for quantization groups of 64 columns.
#include "decode.hpp"

namespace mc {
template hipError_t launch_decode<2, true>(const LayerArgs&, const DecodeArgs&, hipStream_t);
template hipError_t launch_decode<2, false>(const LayerArgs&, const DecodeArgs&, hipStream_t);
}  // namespace mc
