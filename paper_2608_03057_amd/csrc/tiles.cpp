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

const PackedTileOps &ops_ptile_256x256_k128_w8();
const PackedTileOps &ops_ptile_256x256_k64_w8();
const PackedTileOps &ops_ptile_128x256_k128_w4();
const PackedTileOps &ops_ptile_128x256_k64_w4();
const PackedTileOps &ops_ptile_256x128_k64_w4();
const PackedTileOps &ops_ptile_128x128_k64_w4();
const PackedTileOps &ops_ptile_64x64_k128_w4();

using PackedOpsFn = const PackedTileOps &(*)();
static const PackedOpsFn kPackedTiles[PTILE_COUNT] = {
    &ops_ptile_256x256_k128_w8,
    &ops_ptile_256x256_k64_w8,
    &ops_ptile_128x256_k128_w4,
    &ops_ptile_128x256_k64_w4,
    &ops_ptile_256x128_k64_w4,
    &ops_ptile_128x128_k64_w4,
    &ops_ptile_64x64_k128_w4};

const PackedTileOps &packed_tile_ops(int tile)
{
    if (tile < 0 || tile >= PTILE_COUNT)
        tile = PTILE_128x128_K64_W4;
    return kPackedTiles[tile]();
}

}  // namespace tasq
