// Bit-plane relayout of the stored weight buffer (one-time).
//
// planes[q][kb][n][w] holds bit p = 7 - q of the codes of W[n][128*kb ..]
// (App. G.2: plane p is bit p of the two's-complement code; most significant
// plane first so that the top b planes form one contiguous prefix).  The
// 128 elements of a block split into four sub-steps of 32 (s), each into two
// halves of 16 (h) of four groups (i) of four bytes (c).  Word w = 2h + t
// holds half h of sub-steps 2t and 2t+1; element (s, h, i, c) sits at bit
// (8c + g + p) mod 32 with g = 4(s % 2) + i.  Rotating each plane's word left
// by p puts the b planes' bits of one group g on disjoint positions, so the
// reader merges them with one AND-OR per plane and one rotate right by g
// yields bit p of each of the group's four bytes.
#include "tasq_internal.h"

namespace tasq {

// One thread per output word: reads the 32 codes it covers (zero past K)
// and emits their 8 plane words.
__global__ void k_pack_planes(const int8_t *__restrict__ W, int N, int K, int KB,
                              uint32_t *__restrict__ planes)
{
    const long long words = (long long)KB * N * 4;
    for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < words;
         idx += (long long)gridDim.x * blockDim.x) {
        const int w = (int)(idx & 3);
        const long long rest = idx >> 2;
        const int n = (int)(rest % N);
        const int kb = (int)(rest / N);
        const int h = w >> 1, t = w & 1;
        uint32_t pw[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        const int8_t *row = W + (size_t)n * (size_t)K;
        for (int e = 0; e < 32; ++e) {
            const int sl = e >> 4;                 // which of the word's two sub-steps
            const int i = (e >> 2) & 3, c = e & 3;
            const int j = kb * 128 + 32 * (2 * t + sl) + 16 * h + 4 * i + c;
            const uint32_t v = j < K ? (uint32_t)(uint8_t)row[j] : 0u;
            const int g = 4 * sl + i;
#pragma unroll
            for (int p = 0; p < 8; ++p)
                pw[p] |= ((v >> p) & 1u) << ((8 * c + g + p) & 31);
        }
#pragma unroll
        for (int p = 0; p < 8; ++p)
            planes[(size_t)(7 - p) * (size_t)words + (size_t)idx] = pw[p];
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
