// Masked linear for skinny activations (M <= 64): weight-streaming kernels.
//
// With few activation rows a layer reads each weight once and does little
// arithmetic per byte, so its time is the weight stream.  Three sources of
// the weight operand:
//   * int8 rows [N][K], masked with one v_and_b32 per 4 weights;
//   * the packed buffer (tasq_pack_weights), 1 KB per 32 x 32 fragment;
//   * bit planes, reading only the top b planes (App. G.2; the dropped
//     planes are never fetched): b/8 byte per weight, rebuilt into the
//     two's-complement bytes of W_b in registers (one AND-OR per plane and
//     one rotate per 4 weights, from the rotated plane words).
// A workgroup owns 32 output channels; its W waves take interleaved 128-byte
// K blocks and compute acc^T = W_b X^T with v_mfma_i32_16x16x64_i8, 16
// channels x 16 tokens x 64 K per instruction (A = weight rows, B = one tile
// of up to 16 activation rows; MT tiles cover M <= 16 MT).  The waves' exact
// int32 partial sums are added through LDS in a fixed order and the
// workgroup writes acc and y = acc * sx * sw[n] + bias[n] itself: one launch,
// no atomics, no workspace.  The grouped form covers every layer of a
// denoising step in one launch, its b taken from the (layer, stage) table,
// with W = 4 waves per workgroup: nine or 36 K blocks (1152- and 4608-deep
// layers) keep every wave busy to the end, where 8 waves leave 7 of them
// idle through the second of a 1152-deep layer's two rounds.  A single
// layer, with few workgroups, keeps W = 8 for more loads in flight.
#include "gemm_core.h"
#include "gemm_packed.h"

namespace tasq {

namespace {

constexpr int SK_WAVES_SINGLE = 8;    // waves per workgroup, one layer per launch
constexpr int SK_WAVES_GROUPED = 4;   // waves per workgroup, a schedule step per launch
constexpr int SK_KBLK = 128;          // K bytes per block (two 64-wide MFMA steps)
constexpr int SK_PAD = 65;            // LDS row pitch (ints) of the reduction buffer

enum SkinnySource : int { SRC_ROWS = 0, SRC_PACKED = 1, SRC_PLANES = 2 };

// Weight stream of output channels 32*nb .. 32*nb+31 of layer d at b bits,
// MT 16-token tiles: each wave's int32 partial sums go to red.  BP is b as a
// compile-time count for the plane source (one copy of the loop per b, so
// the plane loop has no branches), 0 otherwise.
//
// Operand order.  Lane l feeds row r = l % 16 of both operands (a channel of
// the A operand, a token of the B operand) with 16 consecutive K bytes; a
// wave takes both 16-channel halves f of the block (channels n0 + 16 f + r).
// Any assignment of a block's K bytes to (lane group, step) gives the same
// sums when both operands follow it; lane group j = l / 16 takes bytes
// kj + 32 t at step t = 0, 1, kj = 64 (j & 1) + 16 (j >> 1).  These are
// exactly the codes of plane word j of the block (groups 0-3 of the word:
// t = 0, groups 4-7: t = 1), and the plane layout stores word j of channels
// n0 + r and n0 + 16 + r side by side, so a lane reads both halves' word
// with one 8-byte load per plane: a wave reads 512 contiguous bytes per
// plane and block, and a workgroup's top b planes are one contiguous run.
// Register v of accumulator (f, mt) of lane l is channel n0 + 16 f +
// 4 (l / 16) + v, token 16 mt + l % 16.
// Packed weights are read once per step in whole 16-byte MFMA fragments:
// non-temporal loads (about 3.5% shorter step at 16 tokens; the row and
// plane streams measured slower with them).
__device__ __forceinline__ v4i ld16_nt(rsrc_t r, uint32_t off)
{
    return __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2));
}

template <int SRC, int MT, int BP, int W>
__device__ __forceinline__ void skinny_stream(const LayerDesc &d, int b, int nb, int *red)
{
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int r = lane & 15, j = lane >> 4;
    const int n0 = nb * 32;
    const int nkb = (d.K + SK_KBLK - 1) / SK_KBLK;
    const uint32_t kj = 64u * (uint32_t)(j & 1) + 16u * (uint32_t)(j >> 1);

    const rsrc_t rX = make_rsrc(d.X, (uint32_t)d.M * (uint32_t)d.K);
    uint32_t offX[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int m = 16 * mt + r;
        offX[mt] = m < d.M ? (uint32_t)m * (uint32_t)d.K + kj : kOOB;
    }
    const int msk = (int)keep_mask_dword(b);

    v4i acc[2][MT];
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            acc[f][mt] = zero4();

    rsrc_t rW;
    uint32_t offW[2];
    uint32_t plane_stride = 0;
    if constexpr (SRC == SRC_PLANES) {
        // words planes[nb][q][kb][r][j][0..1]
        plane_stride = (uint32_t)nkb * 512u;
        rW = make_rsrc(d.P, (uint32_t)planes_bytes(d.N, d.K));
        offW[0] = (uint32_t)nb * 8u * plane_stride + (uint32_t)(4 * r + j) * 8u;
        offW[1] = 0;
    } else if constexpr (SRC == SRC_PACKED) {
        // unit (nb, 4 kb + 2 (j & 1) + t), row 16 f + r of lane half j >> 1
        rW = make_rsrc(d.Wp, (uint32_t)packed_weight_bytes(d.N, d.K));
        const uint32_t o = (uint32_t)nb * (uint32_t)(4 * nkb) * 1024u + 2048u * (uint32_t)(j & 1) +
                           (uint32_t)(32 * (j >> 1) + r) * 16u;
        offW[0] = o;
        offW[1] = o + 256u;
    } else {
        rW = make_rsrc(d.W, (uint32_t)d.N * (uint32_t)d.K);
#pragma unroll
        for (int f = 0; f < 2; ++f) {
            const int n = n0 + 16 * f + r;
            offW[f] = n < d.N ? (uint32_t)n * (uint32_t)d.K + kj : kOOB;
        }
    }

    // One K block's operands: every load of the block is issued before any
    // is used.  Latency is covered by the other waves of the CU (8 per SIMD
    // with one token tile) rather than by a second buffer, except in the
    // grouped packed stream (below).
    struct Block {
        v2i pw[8];
        v4i w[2][2];
        v4i x[2][MT];
    };
    auto load = [&](int kb, Block &bl) {
        const uint32_t k0 = (uint32_t)kb * SK_KBLK;
        if constexpr (SRC == SRC_PLANES) {
            const uint32_t base = offW[0] + (uint32_t)kb * 512u;
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                bl.pw[q] = v2i{0, 0};
                if (q < BP)
                    bl.pw[q] = ld8(rW, base + (uint32_t)q * plane_stride);
            }
        } else {
#pragma unroll
            for (int f = 0; f < 2; ++f)
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    if constexpr (SRC == SRC_PACKED)
                        bl.w[f][t] = ld16_nt(rW, offW[f] + (uint32_t)(4 * kb + t) * 1024u);
                    else
                        bl.w[f][t] = ld16(rW, offW[f] + k0 + 32u * t);
                }
        }
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                bl.x[t][mt] = ld16(rX, offX[mt] + k0 + 32u * t);
    };
    // Step t, half f: the weight fragment is rebuilt (planes) or masked
    // (int8) and consumed at once, so only one fragment is live.
    auto compute = [&](int kb, const Block &bl) {
        const uint32_t k0 = (uint32_t)kb * SK_KBLK;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int f = 0; f < 2; ++f) {
                v4i wq = zero4();
                if constexpr (SRC == SRC_PLANES) {
                    uint32_t m0 = 0, m1 = 0, m2 = 0, m3 = 0;
                    const int g0 = 4 * t;
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        if (q < BP) {
                            const uint32_t w = (uint32_t)(f == 0 ? bl.pw[q].x : bl.pw[q].y);
                            const int p = 7 - q;
                            m0 = plane_bits(w, g0 + 0, p, m0);
                            m1 = plane_bits(w, g0 + 1, p, m1);
                            m2 = plane_bits(w, g0 + 2, p, m2);
                            m3 = plane_bits(w, g0 + 3, p, m3);
                        }
                    }
                    wq = v4i{(int)plane_place(m0, g0 + 0), (int)plane_place(m1, g0 + 1),
                             (int)plane_place(m2, g0 + 2), (int)plane_place(m3, g0 + 3)};
                } else {
                    wq = bl.w[f][t];
                    wq.x &= msk;
                    wq.y &= msk;
                    wq.z &= msk;
                    wq.w &= msk;
                    // Columns past K: zero the weights (row-major loads there
                    // may hold the next row; packed and plane layouts are zero).
                    if (SRC == SRC_ROWS && k0 + kj + 32u * t >= (uint32_t)d.K)
                        wq = zero4();
                }
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    acc[f][mt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wq, bl.x[t][mt],
                                                                         acc[f][mt], 0, 0, 0);
            }
    };

    if constexpr (SRC == SRC_PACKED && MT == 1 && W == SK_WAVES_GROUPED) {
        // The grouped packed stream with one token tile also keeps the next K
        // block's loads in flight while it computes the current one (6
        // waves per SIMD instead of 8): at 16 tokens its step is 6% shorter.
        // The plane stream needs all 8 waves to hide its rebuild (a second
        // buffer made it 7-10% slower), the row stream gains nothing, and
        // the single-layer launch's 8 waves hold one or two K blocks each.
        Block b0, b1;
        int kb = wave;
        if (kb < nkb)
            load(kb, b0);
        while (kb < nkb) {
            const int k1 = kb + W;
            if (k1 < nkb)
                load(k1, b1);
            compute(kb, b0);
            if (k1 >= nkb)
                break;
            const int k2 = k1 + W;
            if (k2 < nkb)
                load(k2, b0);
            compute(k1, b1);
            kb = k2;
        }
    } else {
        for (int kb = wave; kb < nkb; kb += W) {
            Block bl;
            load(kb, bl);
            compute(kb, bl);
        }
    }

#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                red[(((wave * 2 + f) * MT + mt) * 4 + v) * SK_PAD + lane] = acc[f][mt][v];
}

// Ints of a workgroup's reduction buffer.
template <int MT, int W>
constexpr int skinny_red_ints() { return W * 2 * MT * 4 * SK_PAD; }

// Index in red of wave w's partial sum of token row, channel n0 + col.
template <int MT>
__device__ __forceinline__ int skinny_red_index(int w, int row, int col)
{
    const int f = col >> 4, c = col & 15;
    return (((w * 2 + f) * MT + (row >> 4)) * 4 + (c & 3)) * SK_PAD + 16 * (c >> 2) + (row & 15);
}

// Output channels 32*nb .. 32*nb+31 of layer d at b bits: the weight stream,
// then the fixed-order reduction of the waves' partials and the epilogue.
template <int SRC, int MT, int W>
__device__ __forceinline__ void skinny_block(const LayerDesc &d, int b, int nb, int *red)
{
    if constexpr (SRC == SRC_PLANES) {
        switch (b) {
        case 1: skinny_stream<SRC, MT, 1, W>(d, b, nb, red); break;
        case 2: skinny_stream<SRC, MT, 2, W>(d, b, nb, red); break;
        case 3: skinny_stream<SRC, MT, 3, W>(d, b, nb, red); break;
        case 4: skinny_stream<SRC, MT, 4, W>(d, b, nb, red); break;
        case 5: skinny_stream<SRC, MT, 5, W>(d, b, nb, red); break;
        case 6: skinny_stream<SRC, MT, 6, W>(d, b, nb, red); break;
        case 7: skinny_stream<SRC, MT, 7, W>(d, b, nb, red); break;
        default: skinny_stream<SRC, MT, 8, W>(d, b, nb, red); break;
        }
    } else {
        skinny_stream<SRC, MT, 0, W>(d, b, nb, red);
    }
    __syncthreads();

    const int tid = threadIdx.x;
    const int n0 = nb * 32;

    // Thread t writes channel n0 + t%32 of tokens t/32 + RP*i: 32 threads
    // cover one 128-byte output row segment.
    constexpr int RP = 2 * W;               // rows per pass
    const int col = tid & 31;
    const int nn = n0 + col;
    float scale = 0.f, bias = 0.f, corr = 0.f;
    if (nn < d.N && d.y) {
        if (d.act) {
            scale = d.act[0] * d.sw[nn];
            corr = (128.0f - d.act[1]) * (float)d.colsums[(b - 1) * d.N + nn];
        } else {
            scale = d.sx * d.sw[nn];
        }
        if (d.bias)
            bias = d.bias[nn];
    }
#pragma unroll
    for (int i = 0; i < (16 * MT + RP - 1) / RP; ++i) {
        const int row = (tid >> 5) + RP * i;
        if (row >= d.M || nn >= d.N)
            continue;
        int sum = 0;
#pragma unroll
        for (int w = 0; w < W; ++w)
            sum += red[skinny_red_index<MT>(w, row, col)];
        const size_t o = (size_t)row * (size_t)d.N + (size_t)nn;
        if (d.acc)
            d.acc[o] = sum;
        if (d.y) {
            // Low-rank branch (T U^T)[row][nn]: a rank <= 32 dot product in
            // fp32 (U in bfloat16).
            float lr = 0.f;
            if (d.lr_T) {
                const float *t = d.lr_T + (size_t)row * (size_t)d.lr_r;
                const uint16_t *u = d.lr_U + (size_t)nn * (size_t)d.lr_r;
                for (int q = 0; q < d.lr_r; ++q)
                    lr = fmaf(t[q], __uint_as_float((uint32_t)u[q] << 16), lr);
            }
            // Weight zero point: (128 - z_n) times the row's activation sum
            // (plus K (128 - z_x) for asymmetric codes).
            if (d.wz) {
                const float R = (float)d.xrs[row] +
                                (d.act ? (float)d.K * (128.0f - d.act[1]) : 0.0f);
                lr += (128.0f - d.wz[nn]) * scale * R;
            }
            d.y[o] = ((float)sum + corr) * scale + bias + lr;
        }
    }
}

// Occupancy: with one token tile the streaming loop fits 64 VGPRs, 8 waves
// per SIMD (32 waves per CU: four 8-wave or eight 4-wave workgroups), or
// 80 for the packed stream's two K blocks in flight (6 waves); each further
// tile adds 16 accumulator and activation registers.  The epilogue's
// optional terms must not push a form past its count.
template <int SRC, int MT, bool GROUPED>
constexpr int skinny_waves_per_eu()
{
    return MT == 1 ? (SRC == SRC_PACKED && GROUPED ? 6 : 8) : MT == 2 ? 6 : MT == 3 ? 5 : 4;
}

template <int SRC, int MT>
__global__ void __launch_bounds__(SK_WAVES_SINGLE * 64)
__attribute__((amdgpu_waves_per_eu(skinny_waves_per_eu<SRC, MT, false>()))) k_skinny(LayerDesc d)
{
    __shared__ int red[skinny_red_ints<MT, SK_WAVES_SINGLE>()];
    skinny_block<SRC, MT, SK_WAVES_SINGLE>(d, d.bits, blockIdx.x, red);
}

// One launch per denoising step over every layer's 32-channel blocks;
// d.tile_begin is the layer's first block.
template <int SRC, int MT>
__global__ void __launch_bounds__(SK_WAVES_GROUPED * 64)
__attribute__((amdgpu_waves_per_eu(skinny_waves_per_eu<SRC, MT, true>())))
k_skinny_grouped(const LayerDesc *__restrict__ descs, int L, const uint8_t *table, int S, int stage)
{
    __shared__ int red[skinny_red_ints<MT, SK_WAVES_GROUPED>()];
    const int t = blockIdx.x;
    int lo = 0, hi = L - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (descs[mid].tile_begin <= t)
            lo = mid;
        else
            hi = mid - 1;
    }
    const LayerDesc d = descs[lo];
    skinny_block<SRC, MT, SK_WAVES_GROUPED>(d, table[d.layer * S + stage],
                                            t - d.tile_begin + d.tile_first, red);
}

// Token tiles of 16 rows for M rows (M <= 64).
template <int SRC, template <int, int> class Launch, typename... Args>
hipError_t dispatch_tiles(int m, Args... args)
{
    if (m > 48)
        return Launch<SRC, 4>::run(args...);
    if (m > 32)
        return Launch<SRC, 3>::run(args...);
    if (m > 16)
        return Launch<SRC, 2>::run(args...);
    return Launch<SRC, 1>::run(args...);
}

template <int SRC, int MT>
struct LaunchSingle {
    static hipError_t run(const LayerDesc &d, hipStream_t stream)
    {
        const unsigned grid = (unsigned)((d.N + 31) / 32);
        hipLaunchKernelGGL((k_skinny<SRC, MT>), dim3(grid), dim3(SK_WAVES_SINGLE * 64), 0, stream,
                           d);
        return hipGetLastError();
    }
};

template <int SRC, int MT>
struct LaunchGrouped {
    static hipError_t run(const LayerDesc *d_descs, int L, int total, const uint8_t *d_table,
                          int S, int stage, hipStream_t stream)
    {
        hipLaunchKernelGGL((k_skinny_grouped<SRC, MT>), dim3((unsigned)total),
                           dim3(SK_WAVES_GROUPED * 64), 0, stream, d_descs, L, d_table, S,
                           stage);
        return hipGetLastError();
    }
};

template <int SRC>
hipError_t launch_single_src(const LayerDesc &d, hipStream_t stream)
{
    return dispatch_tiles<SRC, LaunchSingle>(d.M, d, stream);
}

template <int SRC>
hipError_t launch_grouped_src(const LayerDesc *d_descs, int L, int total, int max_m,
                              const uint8_t *d_table, int S, int stage, hipStream_t stream)
{
    return dispatch_tiles<SRC, LaunchGrouped>(max_m, d_descs, L, total, d_table, S, stage, stream);
}

}  // namespace

hipError_t launch_skinny(const LayerDesc &d, SkinnyWeights src, hipStream_t stream)
{
    if (d.M > kSkinnyMaxM || d.N <= 0 || d.M <= 0)
        return hipErrorInvalidValue;
    switch (src) {
    case SKINNY_PLANES: return launch_single_src<SRC_PLANES>(d, stream);
    case SKINNY_PACKED: return launch_single_src<SRC_PACKED>(d, stream);
    default: return launch_single_src<SRC_ROWS>(d, stream);
    }
}

hipError_t launch_skinny_grouped(const LayerDesc *d_descs, int L, int total_blocks, int max_m,
                                 SkinnyWeights src, const uint8_t *d_table, int S, int stage,
                                 hipStream_t stream)
{
    if (max_m > kSkinnyMaxM)
        return hipErrorInvalidValue;
    switch (src) {
    case SKINNY_PLANES:
        return launch_grouped_src<SRC_PLANES>(d_descs, L, total_blocks, max_m, d_table, S, stage,
                                              stream);
    case SKINNY_PACKED:
        return launch_grouped_src<SRC_PACKED>(d_descs, L, total_blocks, max_m, d_table, S, stage,
                                              stream);
    default:
        return launch_grouped_src<SRC_ROWS>(d_descs, L, total_blocks, max_m, d_table, S, stage,
                                            stream);
    }
}

}  // namespace tasq
