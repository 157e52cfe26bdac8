// Masked int8 GEMM instantiated for the 64x64 tile, 4 waves (32x32 per wave), BK 128, 2 K tiles in flight.
#include "gemm_core.h"

namespace tasq {
using TileCfg = Cfg<64, 64, 128, 2, 2, 2, 4>;
TASQ_DEFINE_TILE(ops_tile_64x64_k128_w4_pf2, TileCfg)
}  // namespace tasq
