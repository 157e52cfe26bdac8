// Masked linear for skinny activations (M <= 64): weight-streaming kernels.
//
// With few activation rows a layer reads each weight once and does little
// arithmetic per byte, so its time is the weight stream.  Three sources of
// the weight operand:
//   * int8 rows [N][K], masked with one v_and_b32 per 4 weights;
//   * the packed buffer (tasq_pack_weights): each 32 x 32 fragment is one
//     contiguous 1 KB, so a wave's weight loads are fully coalesced;
//   * bit planes, reading only the top b planes (App. G.2; the dropped
//     planes are never fetched): b/8 byte per weight, rebuilt into the
//     two's-complement bytes of W_b in registers (one AND-OR per plane and
//     one rotate per 4 weights, from the rotated plane words).
// A workgroup owns 32 output channels; its 8 waves take interleaved
// 128-byte K blocks and compute acc^T = W_b X^T with v_mfma_i32_32x32x32_i8
// (A = 32 weight rows, B = up to 32 activation rows per m-tile).  The waves'
// exact int32 partial sums are added through LDS in a fixed order and the
// workgroup writes acc and y = acc * sx * sw[n] + bias[n] itself: one launch,
// no atomics, no workspace.  The grouped form covers every layer of a
// denoising step in one launch, its b taken from the (layer, stage) table.
#include "gemm_core.h"
#include "gemm_packed.h"

namespace tasq {

namespace {

constexpr int SK_WAVES = 8;
constexpr int SK_KBLK = 128;          // K bytes per block (four 32-wide MFMA steps)
constexpr int SK_PAD = 65;            // LDS row pitch (ints) of the reduction buffer

enum SkinnySource : int { SRC_ROWS = 0, SRC_PACKED = 1, SRC_PLANES = 2 };

// Weight stream of output channels 32*nb .. 32*nb+31 of layer d at b bits:
// each wave's int32 partial sums go to red, SK_WAVES * MT * 16 rows of
// SK_PAD ints.  BP is b as a compile-time count for the plane source (one
// copy of the loop per b, so the plane loop has no branches), 0 otherwise.
template <int SRC, int MT, int BP>
__device__ __forceinline__ void skinny_stream(const LayerDesc &d, int b, int nb, int *red)
{
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int h = lane >> 5, r = lane & 31;
    const int n0 = nb * 32;
    const int n = n0 + r;
    const int nkb = (d.K + SK_KBLK - 1) / SK_KBLK;

    const rsrc_t rX = make_rsrc(d.X, (uint32_t)d.M * (uint32_t)d.K);
    uint32_t offX[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int m = 32 * mt + r;
        offX[mt] = m < d.M ? (uint32_t)m * (uint32_t)d.K + 16 * h : kOOB;
    }
    const int msk = (int)keep_mask_dword(b);

    v16i acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
        acc[mt] = v16i{};

    rsrc_t rW;
    uint32_t offW;
    uint32_t plane_stride = 0;
    if constexpr (SRC == SRC_PLANES) {
        // words planes[q][kb][n][2h], [2h + 1]: this lane half's 16 weights
        // of sub-steps 0, 1 and of 2, 3
        plane_stride = (uint32_t)nkb * (uint32_t)d.N * 16u;
        rW = make_rsrc(d.P, 8u * plane_stride);
        offW = n < d.N ? (uint32_t)n * 16u + 8u * (uint32_t)h : kOOB;
    } else if constexpr (SRC == SRC_PACKED) {
        // unit (nb, 4*kb + s), this lane's 16 bytes
        const int NB = (d.N + 31) / 32;
        rW = make_rsrc(d.Wp, (uint32_t)packed_weight_bytes(d.N, d.K));
        offW = nb < NB ? (uint32_t)nb * (uint32_t)(4 * nkb) * 1024u + (uint32_t)lane * 16u : kOOB;
    } else {
        rW = make_rsrc(d.W, (uint32_t)d.N * (uint32_t)d.K);
        offW = n < d.N ? (uint32_t)n * (uint32_t)d.K + 16 * h : kOOB;
    }

    // One K block's operands: every load of the block is issued before any
    // is used.  Latency is covered by the other waves of the CU rather than
    // by a second buffer, which would halve the waves that fit.  Planes: one
    // 8-byte load per plane (a wave reads 32 rows x 16 contiguous bytes).
    struct Block {
        v4i w[4];
        v2i pw[8];
        v4i x[4][MT];
    };
    auto load = [&](int kb, Block &bl) {
        const uint32_t k0 = (uint32_t)kb * SK_KBLK;
        if constexpr (SRC == SRC_PLANES) {
            const uint32_t base = offW + (uint32_t)kb * (uint32_t)d.N * 16u;
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                bl.pw[q] = v2i{0, 0};
                if (q < BP)
                    bl.pw[q] = ld8(rW, base + (uint32_t)q * plane_stride);
            }
        } else {
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                if constexpr (SRC == SRC_PACKED)
                    bl.w[s] = ld16(rW, offW + (uint32_t)(4 * kb + s) * 1024u);
                else
                    bl.w[s] = ld16(rW, offW + k0 + 32 * s);
            }
        }
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                bl.x[s][mt] = ld16(rX, offX[mt] + k0 + 32 * s);
    };
    // Sub-step s of a block: weight fragment rebuilt (planes) or masked
    // (int8) and consumed at once, so only one fragment is live.
    auto compute = [&](int kb, const Block &bl) {
        const uint32_t k0 = (uint32_t)kb * SK_KBLK;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            v4i wq = zero4();
            if constexpr (SRC == SRC_PLANES) {
                // groups 4(s % 2) .. +3 of word s / 2 of each plane
                uint32_t m0 = 0, m1 = 0, m2 = 0, m3 = 0;
                const int g0 = 4 * (s & 1);
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    if (q < BP) {
                        const uint32_t w = (uint32_t)(s < 2 ? bl.pw[q].x : bl.pw[q].y);
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
                wq = bl.w[s];
                wq.x &= msk;
                wq.y &= msk;
                wq.z &= msk;
                wq.w &= msk;
                // Columns past K: zero the weights (row-major loads there may
                // hold the next row; packed and plane layouts are zero).
                if (SRC == SRC_ROWS && k0 + 32 * s + 16 * h >= (uint32_t)d.K)
                    wq = zero4();
            }
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                acc[mt] = __builtin_amdgcn_mfma_i32_32x32x32_i8(wq, bl.x[s][mt], acc[mt], 0, 0, 0);
        }
    };

    for (int kb = wave; kb < nkb; kb += SK_WAVES) {
        Block bl;
        load(kb, bl);
        compute(kb, bl);
    }

    // Each wave's partial block: register v of lane l is channel
    // 8*(v/4) + 4*(l/32) + v%4, token l%32.
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int v = 0; v < 16; ++v)
            red[((wave * MT + mt) * 16 + v) * SK_PAD + lane] = acc[mt][v];
}

// Output channels 32*nb .. 32*nb+31 of layer d at b bits: the weight stream,
// then the fixed-order reduction of the waves' partials and the epilogue.
template <int SRC, int MT>
__device__ __forceinline__ void skinny_block(const LayerDesc &d, int b, int nb, int *red)
{
    if constexpr (SRC == SRC_PLANES) {
        switch (b) {
        case 1: skinny_stream<SRC, MT, 1>(d, b, nb, red); break;
        case 2: skinny_stream<SRC, MT, 2>(d, b, nb, red); break;
        case 3: skinny_stream<SRC, MT, 3>(d, b, nb, red); break;
        case 4: skinny_stream<SRC, MT, 4>(d, b, nb, red); break;
        case 5: skinny_stream<SRC, MT, 5>(d, b, nb, red); break;
        case 6: skinny_stream<SRC, MT, 6>(d, b, nb, red); break;
        case 7: skinny_stream<SRC, MT, 7>(d, b, nb, red); break;
        default: skinny_stream<SRC, MT, 8>(d, b, nb, red); break;
        }
    } else {
        skinny_stream<SRC, MT, 0>(d, b, nb, red);
    }
    __syncthreads();

    const int tid = threadIdx.x;
    const int n0 = nb * 32;

    // Thread t writes channel n0 + t%32 of tokens t/32 + 16*i: 32 threads
    // cover one 128-byte output row segment.
    const int col = tid & 31;
    const int nn = n0 + col;
    const int vv = 4 * (col >> 3) + (col & 3);
    const int lh = 32 * ((col & 7) >> 2);
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
    for (int i = 0; i < 2 * MT; ++i) {
        const int row = (tid >> 5) + 16 * i;
        if (row >= d.M || nn >= d.N)
            continue;
        const int mt = row >> 5;
        const int ln = (row & 31) + lh;
        int sum = 0;
#pragma unroll
        for (int w = 0; w < SK_WAVES; ++w)
            sum += red[((w * MT + mt) * 16 + vv) * SK_PAD + ln];
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

// Occupancy: with one 32-token block (MT = 1) the streaming loop fits 80
// VGPRs, i.e. 6 waves per SIMD (three 8-wave workgroups per CU); the
// epilogue's optional terms must not push it past that.
template <int MT>
constexpr int skinny_waves_per_eu() { return MT == 1 ? 6 : 4; }

template <int SRC, int MT>
__global__ void __launch_bounds__(SK_WAVES * 64)
__attribute__((amdgpu_waves_per_eu(skinny_waves_per_eu<MT>()))) k_skinny(LayerDesc d)
{
    __shared__ int red[SK_WAVES * MT * 16 * SK_PAD];
    skinny_block<SRC, MT>(d, d.bits, blockIdx.x, red);
}

// One launch per denoising step over every layer's 32-channel blocks;
// d.tile_begin is the layer's first block.
template <int SRC, int MT>
__global__ void __launch_bounds__(SK_WAVES * 64)
__attribute__((amdgpu_waves_per_eu(skinny_waves_per_eu<MT>())))
k_skinny_grouped(const LayerDesc *__restrict__ descs, int L, const uint8_t *table, int S, int stage)
{
    __shared__ int red[SK_WAVES * MT * 16 * SK_PAD];
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
    skinny_block<SRC, MT>(d, table[d.layer * S + stage], t - d.tile_begin + d.tile_first, red);
}

template <int SRC>
hipError_t launch_single_src(const LayerDesc &d, hipStream_t stream)
{
    const unsigned grid = (unsigned)((d.N + 31) / 32);
    if (d.M > 32)
        hipLaunchKernelGGL((k_skinny<SRC, 2>), dim3(grid), dim3(SK_WAVES * 64), 0, stream, d);
    else
        hipLaunchKernelGGL((k_skinny<SRC, 1>), dim3(grid), dim3(SK_WAVES * 64), 0, stream, d);
    return hipGetLastError();
}

template <int SRC>
hipError_t launch_grouped_src(const LayerDesc *d_descs, int L, int total, int max_m,
                              const uint8_t *d_table, int S, int stage, hipStream_t stream)
{
    if (max_m > 32)
        hipLaunchKernelGGL((k_skinny_grouped<SRC, 2>), dim3((unsigned)total), dim3(SK_WAVES * 64),
                           0, stream, d_descs, L, d_table, S, stage);
    else
        hipLaunchKernelGGL((k_skinny_grouped<SRC, 1>), dim3((unsigned)total), dim3(SK_WAVES * 64),
                           0, stream, d_descs, L, d_table, S, stage);
    return hipGetLastError();
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
