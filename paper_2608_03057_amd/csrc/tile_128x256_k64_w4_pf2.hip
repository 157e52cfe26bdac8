// Masked int8 GEMM instantiated for the 128x256 tile, 4 waves (64x128 per wave, two workgroups per CU), BK 64.
#include "gemm_core.h"

namespace tasq {
using TileCfg = Cfg<128, 256, 64, 2, 2, 2, 2>;
TASQ_DEFINE_TILE(ops_tile_128x256_k64_w4_pf2, TileCfg)
}  // namespace tasq
