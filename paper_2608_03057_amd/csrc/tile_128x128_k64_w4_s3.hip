// Masked int8 GEMM instantiated for the 128x128 tile, 4 waves (64x64 per
// wave), BK 64, three LDS stages with cross-tile fragment prefetch.
#include "gemm_core.h"

namespace tasq {
using TileCfg = Cfg<128, 128, 64, 2, 2, 2, 2, 3>;
TASQ_DEFINE_TILE(ops_tile_128x128_k64_w4_s3, TileCfg)
}  // namespace tasq
