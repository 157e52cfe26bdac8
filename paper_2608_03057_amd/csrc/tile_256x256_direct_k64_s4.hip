// Direct-to-LDS masked int8 GEMM, 256x256 tile, 4 waves of 128x128, BK 64, four LDS stages.
#include "gemm_direct.h"

namespace tasq {
using TileCfg = CfgD<64, 4>;
TASQ_DEFINE_DIRECT_TILE(ops_tile_256x256_direct_k64_s4, TileCfg)
}  // namespace tasq
