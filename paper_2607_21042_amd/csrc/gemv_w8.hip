// Decode GEMV launchers for FTTS_W8A16 weights (the kernel template is in gemv_impl.hpp).
#include "gemv_impl.hpp"

namespace ftts {
FTTS_GEMV_INSTANCE(FTTS_W8A16, gemv_w8)
}  // namespace ftts
