// Bit-plane relayout of the stored weight buffer (one-time).
//
// Plane q holds bit p = 7 - q of each code (App. G.2: plane p is bit p of the
// two's-complement code; most significant plane first).  The words of one
// 32-channel block nb are stored together, plane after plane, so the top b
// planes of a block are one contiguous run of b * ceil(K/128) * 512 bytes:
//   planes[nb][q][kb][r][w][f],  channel n = 32 nb + 16 f + r  (r < 16),
// word w < 4 of the 128 codes W[n][128 kb ..].  The 128 codes of a block
// split into four sub-steps of 32 (s), each into two halves of 16 (h) of four
// groups (i) of four bytes (c); word w = 2h + t holds half h of sub-steps 2t
// and 2t+1, element (s, h, i, c) at bit (8c + g + p) mod 32 with
// g = 4(s % 2) + i.  Rotating each plane's word left by p puts the b planes'
// bits of one group g on disjoint positions, so the reader merges them with
// one AND-OR per plane and one rotate right by g yields bit p of each of the
// group's four bytes.  The words of channels n and n + 16 (f = 0, 1) sit side
// by side, so the weight-streaming kernel reads both with one 8-byte load.
// Words of channels past N and codes past K are zero.
#include "tasq_internal.h"

namespace tasq {

// One thread per word position (nb, kb, r, w, f): reads the 32 codes it
// covers and emits their 8 plane words.
__global__ void k_pack_planes(const int8_t *__restrict__ W, int N, int K, int KB,
                              long long positions, uint32_t *__restrict__ planes)
{
    for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < positions;
         idx += (long long)gridDim.x * blockDim.x) {
        const int pos = (int)(idx & 127);          // 8 r + 2 w + f
        const int f = pos & 1, w = (pos >> 1) & 3, r = pos >> 3;
        const long long blk = idx >> 7;            // nb * KB + kb
        const int kb = (int)(blk % KB);
        const long long nb = blk / KB;
        const long long n = 32 * nb + 16 * f + r;
        const int h = w >> 1, t = w & 1;
        uint32_t pw[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        if (n < N) {
            const int8_t *row = W + (size_t)n * (size_t)K;
            for (int e = 0; e < 32; ++e) {
                const int sl = e >> 4;             // which of the word's two sub-steps
                const int i = (e >> 2) & 3, c = e & 3;
                const int j = kb * 128 + 32 * (2 * t + sl) + 16 * h + 4 * i + c;
                const uint32_t v = j < K ? (uint32_t)(uint8_t)row[j] : 0u;
                const int g = 4 * sl + i;
#pragma unroll
                for (int p = 0; p < 8; ++p)
                    pw[p] |= ((v >> p) & 1u) << ((8 * c + g + p) & 31);
            }
        }
#pragma unroll
        for (int p = 0; p < 8; ++p)
            planes[((size_t)(nb * 8 + (7 - p)) * (size_t)KB + (size_t)kb) * 128 + (size_t)pos] =
                pw[p];
    }
}

hipError_t launch_pack_planes(const int8_t *W, int N, int K, uint32_t *planes,
                              hipStream_t stream)
{
    const int KB = (K + 127) / 128;
    const long long positions = (long long)((N + 31) / 32) * KB * 128;
    long long blocks = (positions + 255) / 256;
    if (blocks > 65535)
        blocks = 65535;
    hipLaunchKernelGGL(k_pack_planes, dim3((unsigned)blocks), dim3(256), 0, stream, W, N, K, KB,
                       positions, planes);
    return hipGetLastError();
}

}  // namespace tasq
