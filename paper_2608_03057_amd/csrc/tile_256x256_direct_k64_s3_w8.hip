// Direct-to-LDS masked int8 GEMM, 256x256 tile, 8 waves of 128x64, BK 64, three LDS stages.
#include "gemm_direct.h"

namespace tasq {
using TileCfg = CfgD<64, 3, 4>;
TASQ_DEFINE_DIRECT_TILE(ops_tile_256x256_direct_k64_s3_w8, TileCfg)
}  // namespace tasq
