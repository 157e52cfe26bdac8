// Masked int8 GEMM instantiated for the 256x256 tile, 8 waves, BK 64, 3 K tiles in flight.
#include "gemm_core.h"

namespace tasq {
using TileCfg = Cfg<256, 256, 64, 2, 4, 3, 2>;
TASQ_DEFINE_TILE(ops_tile_256x256_k64_w8_pf3, TileCfg)
}  // namespace tasq
