// Packed-weight masked int8 GEMM instantiated for the 128x256 tile, 4 waves (64x128 per wave), BK 64.
#include "gemm_packed.h"

namespace tasq {
using TileCfg = CfgP<128, 256, 64, 2, 2>;
TASQ_DEFINE_PACKED_TILE(ops_ptile_128x256_k64_w4, TileCfg)
}  // namespace tasq
