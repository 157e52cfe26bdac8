// Masked int8 GEMM instantiated for the 256x128 tile, 4 waves (128x64 per wave, two workgroups per CU), BK 64.
#include "gemm_core.h"

namespace tasq {
using TileCfg = Cfg<256, 128, 64, 2, 2, 2, 2>;
TASQ_DEFINE_TILE(ops_tile_256x128_k64_w4_pf2, TileCfg)
}  // namespace tasq
