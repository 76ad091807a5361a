// prefill_g128.hip -- prefill grouped GEMMs for quantization groups of 128 columns.
#include "prefill.hpp"

namespace mc {
template hipError_t launch_prefill_gemm<1>(const LayerArgs&, const int32_t*, const PrefillTables&,
                                           const PrefillGemm&, bool, hipStream_t);
}  // namespace mc
