// Relayout of the stored 8-bit weight buffer into the MFMA operand order
// read by the packed-weight kernels (one-time, like the bit planes).
//
// Unit (nb, ks) of 1 KB holds, for lane l = 0..63 at bytes 16*l .. 16*l+15,
// W[32*nb + l%32][32*ks + 16*(l/32) .. +15]; units are ordered nb-major,
// KS = 4 * ceil(K / 128) units per 32-row block, and every byte past row N
// or column K is zero.  The codes are copied unchanged: masking to b bits
// happens in the kernels, so this one buffer serves every precision.
#include "tasq_internal.h"

namespace tasq {

// One thread per 16-byte chunk of the packed buffer.
__global__ void k_pack_weights(const int8_t *__restrict__ W, int N, int K, int KS,
                               long long chunks, int8_t *__restrict__ packed)
{
    for (long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x; g < chunks;
         g += (long long)gridDim.x * blockDim.x) {
        const int l = (int)(g & 63);
        const long long unit = g >> 6;
        const int ks = (int)(unit % KS);
        const int nb = (int)(unit / KS);
        const int n = 32 * nb + (l & 31);
        const int k0 = 32 * ks + 16 * (l >> 5);
        uint32_t w[4] = {0, 0, 0, 0};
        if (n < N) {
            const int8_t *row = W + (size_t)n * (size_t)K;
            for (int i = 0; i < 16; ++i)
                if (k0 + i < K)
                    w[i >> 2] |= (uint32_t)(uint8_t)row[k0 + i] << (8 * (i & 3));
        }
        uint32_t *out = reinterpret_cast<uint32_t *>(packed + g * 16);
        out[0] = w[0];
        out[1] = w[1];
        out[2] = w[2];
        out[3] = w[3];
    }
}

hipError_t launch_pack_weights(const int8_t *W, int N, int K, int8_t *packed,
                               hipStream_t stream)
{
    const int KS = (K + 127) / 128 * 4;
    const long long chunks = (long long)((N + 31) / 32) * KS * 64;
    long long blocks = (chunks + 255) / 256;
    if (blocks > 65535)
        blocks = 65535;
    if (blocks < 1)
        return hipSuccess;
    hipLaunchKernelGGL(k_pack_weights, dim3((unsigned)blocks), dim3(256), 0, stream, W, N, K, KS,
                       chunks, packed);
    return hipGetLastError();
}

}  // namespace tasq
