// Masked int8 GEMM with register-fed weights: 256x256 tile, 8 waves of
// 128x64, BK 128, activations staged through LDS.
#include "gemm_bdirect.h"

namespace tasq {
TASQ_DEFINE_BDIRECT_TILE(ops_tile_256x256_bdirect_k128_w8, CfgB)
}  // namespace tasq
