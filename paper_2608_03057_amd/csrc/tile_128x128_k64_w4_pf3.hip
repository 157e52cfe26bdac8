// Masked int8 GEMM instantiated for the 128x128 tile, 4 waves, BK 64, 3 K tiles in flight.
#include "gemm_core.h"

namespace tasq {
using TileCfg = Cfg<128, 128, 64, 2, 2, 3, 3>;
TASQ_DEFINE_TILE(ops_tile_128x128_k64_w4_pf3, TileCfg)
}  // namespace tasq
