// Masked int8 GEMM instantiated for the 128x128 tile, 4 waves (64x64 per wave), BK 128, 2 K tiles in flight.
#include "gemm_core.h"

namespace tasq {
using TileCfg = Cfg<128, 128, 128, 2, 2, 2, 2>;
TASQ_DEFINE_TILE(ops_tile_128x128_k128_w4_pf2, TileCfg)
}  // namespace tasq
