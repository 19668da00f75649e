// Decode GEMV launchers: LayerNorm-fused layers, FTTS_BF16 weights.
#include "gemv_impl.hpp"

namespace ftts {
hipError_t gemv_ln_bf16(int epi, const GemvArgs& a, Tiling t, hipStream_t st) {
    return gemv_dispatch_ln<FTTS_BF16>(epi, a, t, st);
}
}  // namespace ftts
