// Packed-weight masked int8 GEMM instantiated for the 256x256 tile, 8 waves (128x64 per wave),
// BK 128, with the persistent grouped step.
#include "gemm_pers_packed.h"

namespace tasq {
using TileCfg = CfgP<256, 256, 128, 2, 4>;
TASQ_DEFINE_PACKED_TILE_PERS(ops_ptile_256x256_k128_w8, TileCfg)
}  // namespace tasq
