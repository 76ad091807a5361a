// prefill_g32.hip -- prefill grouped GEMMs for quantization groups of 32 columns.
#include "prefill.hpp"

namespace mc {
template hipError_t launch_prefill_gemm<4>(const LayerArgs&, const int32_t*, const PrefillTables&,
                                           const PrefillGemm&, bool, hipStream_t);
}  // namespace mc
