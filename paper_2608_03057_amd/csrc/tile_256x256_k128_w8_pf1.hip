// Masked int8 GEMM instantiated for the 256x256 tile, 8 waves (128x64 per wave), BK 128, 1 K tile in flight;
// its persistent grouped step is the direct-staged one of gemm_pers.h.
#include "gemm_pers.h"

namespace tasq {
using TileCfg = Cfg<256, 256, 128, 2, 4, 1, 2>;
TASQ_DEFINE_TILE_DS(ops_tile_256x256_k128_w8_pf1, TileCfg)
}  // namespace tasq
