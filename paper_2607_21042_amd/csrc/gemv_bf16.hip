// Decode GEMV launchers for FTTS_BF16 weights (the kernel template is in gemv_impl.hpp).
#include "gemv_impl.hpp"

namespace ftts {
FTTS_GEMV_INSTANCE(FTTS_BF16, gemv_bf16)
}  // namespace ftts
