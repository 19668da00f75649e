// Decode GEMV launchers: LayerNorm-fused layers, FTTS_F32 weights.
#include "gemv_impl.hpp"

namespace ftts {
hipError_t gemv_ln_f32(int epi, const GemvArgs& a, Tiling t, hipStream_t st) {
    return gemv_dispatch_ln<FTTS_F32>(epi, a, t, st);
}
}  // namespace ftts
