// Decode GEMV launchers: residual layers, FTTS_F32 weights.
#include "gemv_impl.hpp"

namespace ftts {
hipError_t gemv_res_f32(int epi, const GemvArgs& a, Tiling t, hipStream_t st) {
    return gemv_dispatch_res<FTTS_F32>(epi, a, t, st);
}
}  // namespace ftts
