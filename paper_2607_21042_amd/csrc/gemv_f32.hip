// Decode GEMV launchers for FTTS_F32 weights (the kernel template is in gemv_impl.hpp).
#include "gemv_impl.hpp"

namespace ftts {
FTTS_GEMV_INSTANCE(FTTS_F32, gemv_f32)
}  // namespace ftts
