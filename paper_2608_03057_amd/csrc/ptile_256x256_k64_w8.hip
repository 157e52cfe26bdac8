// Packed-weight masked int8 GEMM instantiated for the 256x256 tile, 8 waves (128x64 per wave), BK 64.
#include "gemm_packed.h"

namespace tasq {
using TileCfg = CfgP<256, 256, 64, 2, 4>;
TASQ_DEFINE_PACKED_TILE(ops_ptile_256x256_k64_w8, TileCfg)
}  // namespace tasq
