// Decode GEMV launchers: LayerNorm-fused layers, FTTS_BF16 weights.
// One weight type per translation unit: the dispatch instantiates every tiling and
// epilogue of gemv_impl.hpp for it, minutes of compilation, so the types build in parallel.
#include "gemv_impl.hpp"

namespace ftts {
hipError_t gemv_ln_bf16(int epi, const GemvArgs& a, Tiling t, hipStream_t st) {
    return gemv_dispatch_ln<FTTS_BF16>(epi, a, t, st);
}
}  // namespace ftts
