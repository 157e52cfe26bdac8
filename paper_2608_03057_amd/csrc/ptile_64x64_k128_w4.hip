// Packed-weight masked int8 GEMM instantiated for the 64x64 tile, 4 waves (32x32 per wave), BK 128.
#include "gemm_packed.h"

namespace tasq {
using TileCfg = CfgP<64, 64, 128, 2, 2, 4>;
TASQ_DEFINE_PACKED_TILE(ops_ptile_64x64_k128_w4, TileCfg)
}  // namespace tasq
