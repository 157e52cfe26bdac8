// Bit-plane relayout of the stored weight buffer (one-time).
//
// planes[q][kb][n][w]: bit 8*(e%4) + e/4 holds bit (7 - q) of element
// W[n][128*kb + 32*w + e] (App. G.2: plane p is bit p of the two's-complement
// code; most significant plane first so that the top b planes form one
// contiguous prefix).  With this order, (word >> s) & 0x01010101 puts the
// bits of elements 4s .. 4s+3 in the low bit of four consecutive bytes.
#include "tasq_internal.h"

namespace tasq {

// One thread per output word: reads the 32 codes it covers (zero past K)
// and emits their 8 plane words.
__global__ void k_pack_planes(const int8_t *__restrict__ W, int N, int K, int KB,
                              uint32_t *__restrict__ planes)
{
    const long long words = (long long)KB * N * 4;
    for (long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x; g < words;
         g += (long long)gridDim.x * blockDim.x) {
        const int w = (int)(g & 3);
        const long long rest = g >> 2;
        const int n = (int)(rest % N);
        const int kb = (int)(rest / N);
        const int j0 = kb * 128 + w * 32;
        uint32_t pw[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        const int8_t *row = W + (size_t)n * (size_t)K;
        for (int i = 0; i < 32; ++i) {
            const int j = j0 + i;
            const uint32_t v = j < K ? (uint32_t)(uint8_t)row[j] : 0u;
            const int pos = 8 * (i & 3) + (i >> 2);
#pragma unroll
            for (int p = 0; p < 8; ++p)
                pw[p] |= ((v >> p) & 1u) << pos;
        }
#pragma unroll
        for (int p = 0; p < 8; ++p)
            planes[(size_t)(7 - p) * (size_t)words + (size_t)g] = pw[p];
    }
}

hipError_t launch_pack_planes(const int8_t *W, int N, int K, uint32_t *planes,
                              hipStream_t stream)
{
    const int KB = (K + 127) / 128;
    const long long words = (long long)KB * N * 4;
    long long blocks = (words + 255) / 256;
    if (blocks > 65535)
        blocks = 65535;
    hipLaunchKernelGGL(k_pack_planes, dim3((unsigned)blocks), dim3(256), 0, stream, W, N, K, KB,
                       planes);
    return hipGetLastError();
}

}  // namespace tasq
