// Internal declarations shared by the HIP kernels and the C-ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace tasq {

enum : int { KIND_LINEAR = 0, KIND_CONV3X3 = 1 };

// One masked GEMM as the kernels see it.  For a grouped schedule launch an
// array of these lives in device memory; single calls pass one by value.
struct LayerDesc {
    const int8_t *X;        // [M][K] (linear) or NHWC [H][Wd][C] (conv)
    const int8_t *W;        // [N][K]
    const uint32_t *P;      // bit planes [8][ceil(K/128)][N][4] or null
    const float *sw;        // [N]
    const float *bias;      // [N] or null
    int32_t *acc;           // [M][N] or null
    float *y;               // [M][N] or null
    float sx;
    int32_t M, N, K;
    int32_t kind;
    int32_t H, Wd, C;
    int32_t bits;           // effective precision b (single calls)
    int32_t tiles_m, tiles_n;
    int32_t tile_begin;     // first tile of this layer in a grouped launch
    int32_t ksplit;         // number of K slices (1 = no split)
    int32_t kslice;         // bytes of K per slice (multiple of the K tile)
    int32_t ws_tile_offset; // first partial-sum tile slot in the workspace
};

// Per-byte keep mask for b effective bits, replicated over the 4 bytes of a
// dword: AND-ing a stored two's-complement code with it clears its 8-b low
// bits, which equals 2^(8-b) * floor(w / 2^(8-b)).
__host__ __device__ inline uint32_t keep_mask_dword(int b)
{
    uint32_t m = (0xFFu << (8 - b)) & 0xFFu;
    return m * 0x01010101u;
}

// Tile configurations the launchers know about.
enum TileId : int {
    TILE_256x256 = 0,
    TILE_128x256 = 1,
    TILE_128x128 = 2,
    TILE_64x64 = 3,
    TILE_COUNT = 4
};

struct TileShape {
    int bm, bn, bk;
};
TileShape tile_shape(int tile);

// Host-side launchers (masked_gemm.hip).
hipError_t launch_single(const LayerDesc &d, int tile, bool aligned, void *ws,
                         hipStream_t stream);
hipError_t launch_grouped(const LayerDesc *d_descs, int L, int total_tiles,
                          const uint8_t *d_table, int S, int stage, int tile,
                          hipStream_t stream);
hipError_t launch_pack_planes(const int8_t *W, int N, int K, uint32_t *planes,
                              hipStream_t stream);
hipError_t launch_bitplane(const LayerDesc &d, bool aligned, hipStream_t stream);

// Bytes of split-K partial sums for a layer (int32 per output of each slice
// except the last, plus one arrival counter per tile).
size_t splitk_workspace_bytes(const LayerDesc &d, int tile);

}  // namespace tasq
