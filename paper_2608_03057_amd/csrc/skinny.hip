// Masked linear for skinny activations (M <= 64): weight-streaming kernels.
//
// With few activation rows the layer reads each weight once and does little
// arithmetic per byte, so its time is the weight stream.  Two sources:
//   * int8 rows, masked with one v_and_b32 per 4 weights: 1 byte per weight;
//   * bit planes, reading only the top b planes (App. G.2; the dropped
//     planes are never fetched): b/8 byte per weight, rebuilt into the
//     two's-complement bytes of W_b in registers (a rotate and an AND-OR
//     place 4 bits of a plane in 4 bytes).
// Each wave owns 32 output channels and a slice of K (no LDS, no barriers),
// computes acc^T = W_b X^T with v_mfma_i32_32x32x32_i8 (A = 32 weight rows,
// B = up to 32 activation rows per m-tile), and adds its int32 partial sums
// into a zeroed int32 buffer with atomics, which is exact and independent of
// the order.  A finishing kernel applies y = acc * sx * sw[n] + bias[n].
#include <algorithm>

#include "gemm_core.h"

namespace tasq {

namespace {

constexpr int SK_KBLK = 128;          // K bytes per plane block (one 16-byte word group)

// The lane half's 16 weights of plane word w (groups 4h .. 4h+3) placed at
// bit `up` of 16 bytes and OR-ed into 4 dwords.
__device__ __forceinline__ void plane_half(uint32_t w, int h, int up, v4i &acc)
{
    acc.x = (int)plane_group(w, 4 * h + 0, up, (uint32_t)acc.x);
    acc.y = (int)plane_group(w, 4 * h + 1, up, (uint32_t)acc.y);
    acc.z = (int)plane_group(w, 4 * h + 2, up, (uint32_t)acc.z);
    acc.w = (int)plane_group(w, 4 * h + 3, up, (uint32_t)acc.w);
}

// One wave: 32 output channels n0..n0+31, K blocks [kb0, kb1) of 128 bytes,
// all m-tiles (MT <= 2 tiles of 32 rows).
template <bool PLANES, int MT>
__global__ void __launch_bounds__(256) k_skinny(LayerDesc d, int blocks_per_wave, int nkb,
                                                int32_t *accbuf)
{
    const int lane = threadIdx.x & 63;
    const int gw = (blockIdx.x * 256 + threadIdx.x) >> 6;     // global wave id
    const int ntiles = (d.N + 31) / 32;
    const int nsl = (nkb + blocks_per_wave - 1) / blocks_per_wave;
    if (gw >= ntiles * nsl)
        return;
    const int nt = gw % ntiles, sl = gw / ntiles;
    const int n0 = nt * 32;
    const int kb0 = sl * blocks_per_wave;
    const int kb1 = min(nkb, kb0 + blocks_per_wave);
    const int h = lane >> 5, r = lane & 31;
    const int n = n0 + r;

    const rsrc_t rX = make_rsrc(d.X, (uint32_t)d.M * (uint32_t)d.K);
    // activation row m = 32*mt + r, lane half h: bytes 16h.. of each 32-k step
    uint32_t offX[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int m = 32 * mt + r;
        offX[mt] = m < d.M ? (uint32_t)m * (uint32_t)d.K + 16 * h : kOOB;
    }
    const int msk = (int)keep_mask_dword(d.bits);

    v16i acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
        acc[mt] = v16i{};

    rsrc_t rW;
    uint32_t offW;
    if constexpr (PLANES) {
        // words planes[q][kb][n][0..3]; plane stride KB*N*16 bytes
        rW = make_rsrc(d.P, (uint32_t)8 * (uint32_t)nkb * (uint32_t)d.N * 16u);
        offW = n < d.N ? (uint32_t)n * 16u : kOOB;
    } else {
        rW = make_rsrc(d.W, (uint32_t)d.N * (uint32_t)d.K);
        offW = n < d.N ? (uint32_t)n * (uint32_t)d.K + 16 * h : kOOB;
    }
    const uint32_t plane_stride = (uint32_t)nkb * (uint32_t)d.N * 16u;
    const int b = d.bits;

    for (int kb = kb0; kb < kb1; ++kb) {
        const uint32_t k0 = (uint32_t)kb * SK_KBLK;
        // weight operand for the 4 sub-steps of this 128-byte K block
        v4i wq[4];
        if constexpr (PLANES) {
            wq[0] = wq[1] = wq[2] = wq[3] = zero4();
            const uint32_t base = offW + (uint32_t)kb * (uint32_t)d.N * 16u;
            for (int q = 0; q < b; ++q) {
                const v4i words = ld16(rW, base + (uint32_t)q * plane_stride);
                const int up = 7 - q;
                plane_half((uint32_t)words.x, h, up, wq[0]);
                plane_half((uint32_t)words.y, h, up, wq[1]);
                plane_half((uint32_t)words.z, h, up, wq[2]);
                plane_half((uint32_t)words.w, h, up, wq[3]);
            }
        } else {
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                v4i v = ld16(rW, offW + k0 + 32 * s);
                v.x &= msk;
                v.y &= msk;
                v.z &= msk;
                v.w &= msk;
                wq[s] = v;
            }
        }
        // columns past K: zero the weights (the activations there may hold
        // the next row)
        if (k0 + SK_KBLK > (uint32_t)d.K) {
#pragma unroll
            for (int s = 0; s < 4; ++s)
                if (k0 + 32 * s + 16 * h >= (uint32_t)d.K)
                    wq[s] = zero4();
        }
#pragma unroll
        for (int s = 0; s < 4; ++s) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const v4i xv = ld16(rX, offX[mt] + k0 + 32 * s);
                acc[mt] = __builtin_amdgcn_mfma_i32_32x32x32_i8(wq[s], xv, acc[mt], 0, 0, 0);
            }
        }
    }
    // acc^T block: register v of lane l is weight row 8*(v/4) + 4*(l/32) + v%4
    // (output channel), column l%32 (activation row)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int m = 32 * mt + (lane & 31);
        if (m >= d.M)
            continue;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int nn = n0 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
            if (nn < d.N)
                atomicAdd(accbuf + (size_t)m * d.N + nn, acc[mt][v]);
        }
    }
}

__global__ void k_fill_zero(int32_t *p, long long n)
{
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (long long)gridDim.x * blockDim.x)
        p[i] = 0;
}

// y = acc * (sx * sw[n]) + bias[n]; acc copied out when it lives in scratch.
__global__ void k_skinny_finish(LayerDesc d, const int32_t *accbuf)
{
    const long long total = (long long)d.M * d.N;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long long)gridDim.x * blockDim.x) {
        const int nn = (int)(i % d.N);
        const int a = accbuf[i];
        if (d.acc && d.acc != accbuf)
            d.acc[i] = a;
        if (d.y)
            d.y[i] = (float)a * (d.sx * d.sw[nn]) + (d.bias ? d.bias[nn] : 0.f);
    }
}

}  // namespace

// K blocks per wave: enough waves (about 8 per SIMD) to cover HBM latency.
static int skinny_blocks_per_wave(const LayerDesc &d)
{
    const int nkb = (d.K + SK_KBLK - 1) / SK_KBLK;
    const long long ntiles = (d.N + 31) / 32;
    const long long target_waves = 256LL * 4 * 8;
    long long slices = (target_waves + ntiles - 1) / ntiles;
    if (slices > nkb)
        slices = nkb;
    if (slices < 1)
        slices = 1;
    return (int)((nkb + slices - 1) / slices);
}

hipError_t launch_skinny(const LayerDesc &d, bool planes, int32_t *accbuf, hipStream_t stream)
{
    if (d.M > 64)
        return hipErrorInvalidValue;
    const long long total = (long long)d.M * d.N;
    const int fill_blocks = (int)std::min<long long>(1024, (total + 255) / 256);
    hipLaunchKernelGGL(k_fill_zero, dim3(fill_blocks), dim3(256), 0, stream, accbuf, total);
    const int nkb = (d.K + SK_KBLK - 1) / SK_KBLK;
    const int bpw = skinny_blocks_per_wave(d);
    const long long waves = (long long)((d.N + 31) / 32) * ((nkb + bpw - 1) / bpw);
    const unsigned grid = (unsigned)((waves + 3) / 4);
    if (nkb > 0) {
        if (planes) {
            if (d.M > 32)
                hipLaunchKernelGGL((k_skinny<true, 2>), dim3(grid), dim3(256), 0, stream, d, bpw,
                                   nkb, accbuf);
            else
                hipLaunchKernelGGL((k_skinny<true, 1>), dim3(grid), dim3(256), 0, stream, d, bpw,
                                   nkb, accbuf);
        } else {
            if (d.M > 32)
                hipLaunchKernelGGL((k_skinny<false, 2>), dim3(grid), dim3(256), 0, stream, d, bpw,
                                   nkb, accbuf);
            else
                hipLaunchKernelGGL((k_skinny<false, 1>), dim3(grid), dim3(256), 0, stream, d, bpw,
                                   nkb, accbuf);
        }
    }
    if (d.y || (d.acc && d.acc != accbuf)) {
        hipLaunchKernelGGL(k_skinny_finish, dim3(fill_blocks), dim3(256), 0, stream, d,
                           (const int32_t *)accbuf);
    }
    return hipGetLastError();
}

}  // namespace tasq
