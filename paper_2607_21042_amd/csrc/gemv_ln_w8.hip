// Decode GEMV launchers: LayerNorm-fused layers, FTTS_W8A16 weights.
#include "gemv_impl.hpp"

namespace ftts {
hipError_t gemv_ln_w8(int epi, const GemvArgs& a, Tiling t, hipStream_t st) {
    return gemv_dispatch_ln<FTTS_W8A16>(epi, a, t, st);
}
}  // namespace ftts
