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
    const int8_t *Wp;       // packed weights (MFMA operand order) or null
    const float *sw;        // [N]
    const float *bias;      // [N] or null
    const float *act;       // asymmetric activation params (alpha at 0, z at 1) or null
    const int32_t *colsums; // [8][N] channel sums of W_b (with act)
    const float *lr_T;      // low-rank branch x~ D^T, fp32 [M][lr_r], or null
    const uint16_t *lr_U;   // its up projection, bfloat16 [N][lr_r]
    const float *wz;        // per-channel weight zero points [N] or null
    const int32_t *xrs;     // row sums of the activation codes [M] (with wz)
    int32_t *acc;           // [M][N] or null
    float *y;               // [M][N] or null
    float sx;
    int32_t M, N, K;
    int32_t kind;
    int32_t H, Wd, C;
    int32_t bits;           // effective precision b (single calls)
    int32_t lr_r;           // rank of the low-rank branch (16 or 32) when lr_T is set
    int32_t tiles_m, tiles_n;
    int32_t tile_begin;     // first work unit of this segment in a grouped launch
    int32_t tile_first;     // the segment's first tile within its layer
    int32_t layer;          // row of the segment's layer in the (layer, stage) table
};

// Per-byte keep mask for b effective bits, replicated over the 4 bytes of a
// dword: AND-ing a stored two's-complement code with it clears its 8-b low
// bits, which equals 2^(8-b) * floor(w / 2^(8-b)).
__host__ __device__ inline uint32_t keep_mask_dword(int b)
{
    uint32_t m = (0xFFu << (8 - b)) & 0xFFu;
    return m * 0x01010101u;
}

struct TileShape {
    int bm, bn, bk;
};

// First work unit of each XCD's run in a persistent launch: XCD x walks
// units begin[x] .. begin[x + 1] - 1 (begin[0] = 0, begin[8] = total).
struct XcdRuns {
    int begin[9];
};

// begin[0] = 0, begin[8] = total and non-decreasing in between.
inline bool xcd_runs_valid(const XcdRuns &r, int total)
{
    if (r.begin[0] != 0 || r.begin[8] != total)
        return false;
    for (int x = 0; x < 8; ++x)
        if (r.begin[x + 1] < r.begin[x])
            return false;
    return true;
}

// Launchers of one tile configuration (one translation unit each).
struct TileOps {
    TileShape shape;
    hipError_t (*single)(const LayerDesc &d, bool aligned, hipStream_t stream);
    hipError_t (*planes)(const LayerDesc &d, bool aligned, hipStream_t stream);
    // One launch over every layer's tiles; any_conv selects the kernel that
    // also handles 3x3 conv layers.
    hipError_t (*grouped)(const LayerDesc *d_descs, int L, int total_tiles,
                          const uint8_t *d_table, int S, int stage, bool any_conv,
                          hipStream_t stream);
    // Split-K partials (aligned operands only) into part[splits][M][N].
    hipError_t (*split)(const LayerDesc &d, int32_t *part, int splits, int kchunk,
                        hipStream_t stream);
    // Persistent form of grouped over linear layers only: wgs_per_xcd
    // workgroups per XCD walk the XCD's run of work units (runs), cut into
    // `parties` parts walked side by side (wgs_per_xcd % parties == 0).
    hipError_t (*persistent)(const LayerDesc *d_descs, int L, int total_tiles,
                             const XcdRuns &runs, const uint8_t *d_table, int S, int stage,
                             int wgs_per_xcd, int parties, hipStream_t stream);
    // The same with the low-rank and weight-zero-point epilogue terms, or
    // null for tiles without one.
    hipError_t (*persistent_extras)(const LayerDesc *d_descs, int L, int total_tiles,
                                    const XcdRuns &runs, const uint8_t *d_table, int S,
                                    int stage, int wgs_per_xcd, int parties, hipStream_t stream);
};

// Sums split-K partials and applies the dequantisation epilogue (splitk.hip).
hipError_t launch_split_finish(const LayerDesc &d, const int32_t *part, int splits,
                               hipStream_t stream);

// Tile configurations, indexed by TileId.
enum TileId : int {
    TILE_256x256_K128_W8_PF1 = 0,  // 256x256 tile, 8 waves (128x64 per wave), BK 128
    TILE_256x256_K64_W8_PF2 = 1,   // 256x256 tile, 8 waves, BK 64, 2 K tiles in flight
    TILE_128x128_K128_W4_PF2 = 2,  // 128x128 tile, 4 waves (64x64 per wave), BK 128
    TILE_64x64_K128_W4_PF2 = 3,    // 64x64 tile, 4 waves (32x32 per wave), BK 128
    TILE_256x128_K64_W4_PF2 = 4,   // 256x128 tile, 4 waves (128x64 per wave), BK 64
    TILE_128x256_K64_W4_PF2 = 5,   // 128x256 tile, 4 waves (64x128 per wave), BK 64
    TILE_COUNT = 6
};
const TileOps &tile_ops(int tile);

// Launchers of one packed-weight tile configuration (gemm_packed.h).
struct PackedTileOps {
    TileShape shape;
    hipError_t (*single)(const LayerDesc &d, bool aligned, hipStream_t stream);
    hipError_t (*grouped)(const LayerDesc *d_descs, int L, int total_tiles,
                          const uint8_t *d_table, int S, int stage, bool any_conv,
                          hipStream_t stream);
    // Persistent grouped step (linear layers, no low-rank or weight-zero-
    // point terms), or null for tiles without one.
    hipError_t (*persistent)(const LayerDesc *d_descs, int L, int total_tiles,
                             const XcdRuns &runs, const uint8_t *d_table, int S, int stage,
                             int wgs_per_xcd, int parties, hipStream_t stream);
};

enum PackedTileId : int {
    PTILE_256x256_K128_W8 = 0,  // 256x256 tile, 8 waves (128x64 per wave), BK 128
    PTILE_256x256_K64_W8 = 1,   // 256x256 tile, 8 waves, BK 64
    PTILE_128x256_K128_W4 = 2,  // 128x256 tile, 4 waves (64x128 per wave), two workgroups per CU
    PTILE_128x256_K64_W4 = 3,   // 128x256 tile, 4 waves, BK 64
    PTILE_256x128_K64_W4 = 4,   // 256x128 tile, 4 waves (128x64 per wave), two workgroups per CU
    PTILE_128x128_K64_W4 = 5,   // 128x128 tile, 4 waves (64x64 per wave)
    PTILE_64x64_K128_W4 = 6,    // 64x64 tile, 4 waves (32x32 per wave), BK 128
    PTILE_COUNT = 7
};
const PackedTileOps &packed_tile_ops(int tile);

// Bytes of the packed weight buffer: 32 * ceil(N/32) * 128 * ceil(K/128).
inline unsigned long long packed_weight_bytes_host(long long N, long long K)
{
    if (N <= 0 || K <= 0)
        return 0;
    return (unsigned long long)((N + 31) / 32) * 32ULL * (unsigned long long)((K + 127) / 128) *
           128ULL;
}

// Bytes of the bit-plane buffer: 8 * 32 * ceil(N/32) * ceil(K/128) * 16.
inline unsigned long long planes_bytes_host(long long N, long long K)
{
    if (N <= 0 || K <= 0)
        return 0;
    return 8ULL * (unsigned long long)((N + 31) / 32) * 32ULL *
           (unsigned long long)((K + 127) / 128) * 16ULL;
}

// Asymmetric 8-bit activation quantizer and the channel sums of the masked
// weight (act_quant.hip).  params: device float[kActHeader + 2 * kActPartials],
// [0] alpha, [1] z on completion, [kActHeader..] partial ranges.
constexpr int kActHeader = 4;
constexpr int kActPartials = 512;

// Largest rank of the 16-bit low-rank branch the epilogues take.
constexpr int kLowrankMaxRank = 32;
// Down projection T = x~ D^T (act_quant.hip); with part set it also writes
// the per-workgroup ranges of x that launch_quantize_activations folds.
// Returns the number of workgroups (partial ranges) through *groups.
hipError_t launch_lowrank_down(const float *x, int M, int K, const uint16_t *D, int r, float *T,
                               uint32_t *part, int *groups, hipStream_t stream);
hipError_t launch_quantize_weights(const float *W, int N, int K, int8_t *Q, float *alpha,
                                   float *z, float *sw, hipStream_t stream);
hipError_t launch_row_sums(const int8_t *X, int M, int K, int32_t *out, hipStream_t stream);
hipError_t launch_quantize_activations_lowrank(const float *x, int M, int K, int8_t *q,
                                               float *params, const uint16_t *D, int r, float *T,
                                               hipStream_t stream);
hipError_t launch_quantize_activations(const float *x, long long n, int8_t *q, float *params,
                                       hipStream_t stream);
// One tensor of a batched activation quantization.
struct ActJob {
    const float *x;
    int M, K;
    int8_t *q;
    float *params;
};
hipError_t launch_quantize_activations_batch(const ActJob *jobs, int n, hipStream_t stream);
hipError_t launch_weight_colsums(const int8_t *W, int N, int K, int32_t *colsums,
                                 hipStream_t stream);

// Packs an [N][K] int8 weight into the MFMA operand order (gemm_packed.h).
hipError_t launch_pack_weights(const int8_t *W, int N, int K, int8_t *packed,
                               hipStream_t stream);

hipError_t launch_pack_planes(const int8_t *W, int N, int K, uint32_t *planes,
                              hipStream_t stream);

// Weight-streaming kernels for M <= 64 (skinny.hip): one workgroup per 32
// output channels reads the weight once from one of three layouts and
// writes acc / y directly.
constexpr int kSkinnyMaxM = 64;
enum SkinnyWeights : int { SKINNY_ROWS = 0, SKINNY_PACKED = 1, SKINNY_PLANES = 2 };
hipError_t launch_skinny(const LayerDesc &d, SkinnyWeights src, hipStream_t stream);
// Grouped step: d_descs[l].tile_begin is layer l's first 32-channel block.
hipError_t launch_skinny_grouped(const LayerDesc *d_descs, int L, int total_blocks, int max_m,
                                 SkinnyWeights src, const uint8_t *d_table, int S, int stage,
                                 hipStream_t stream);

}  // namespace tasq
