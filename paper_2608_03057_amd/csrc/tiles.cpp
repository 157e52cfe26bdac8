// Dispatch table over the tile configurations.
#include "tasq_internal.h"

namespace tasq {

const TileOps &ops_tile_256x256_k128_w8_pf1();
const TileOps &ops_tile_256x256_k64_w8_pf2();
const TileOps &ops_tile_128x128_k128_w4_pf2();
const TileOps &ops_tile_64x64_k128_w4_pf2();
const TileOps &ops_tile_256x128_k64_w4_pf2();
const TileOps &ops_tile_128x256_k64_w4_pf2();

using OpsFn = const TileOps &(*)();
static const OpsFn kTiles[TILE_COUNT] = {
    &ops_tile_256x256_k128_w8_pf1,
    &ops_tile_256x256_k64_w8_pf2,
    &ops_tile_128x128_k128_w4_pf2,
    &ops_tile_64x64_k128_w4_pf2,
    &ops_tile_256x128_k64_w4_pf2,
    &ops_tile_128x256_k64_w4_pf2};

const TileOps &tile_ops(int tile)
{
    if (tile < 0 || tile >= TILE_COUNT)
        tile = TILE_128x128_K128_W4_PF2;
    return kTiles[tile]();
}

}  // namespace tasq
