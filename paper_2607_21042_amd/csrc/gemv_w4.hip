// Decode GEMV launchers for FTTS_W4A16 weights (the kernel template is in gemv_impl.hpp).
#include "gemv_impl.hpp"

namespace ftts {
FTTS_GEMV_INSTANCE(FTTS_W4A16, gemv_w4)
}  // namespace ftts
