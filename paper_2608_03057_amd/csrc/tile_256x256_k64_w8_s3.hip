// Masked int8 GEMM instantiated for the 256x256 tile, 8 waves (128x64 per
// wave), BK 64, three LDS stages with cross-tile fragment prefetch.
#include "gemm_core.h"

namespace tasq {
using TileCfg = Cfg<256, 256, 64, 2, 4, 2, 2, 3>;
TASQ_DEFINE_TILE(ops_tile_256x256_k64_w8_s3, TileCfg)
}  // namespace tasq
