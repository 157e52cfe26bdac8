// Split-K finish: the int32 partials of the K ranges are summed in split
// order (exact, so the result equals the unsplit accumulator bit for bit)
// and the dequantisation epilogue is applied per output element, with every
// term of the tiled epilogue: y = (acc + corr) * scale + bias + (T U^T)[m][n]
// + (128 - z_n) * scale * R[m].
#include "tasq_internal.h"

namespace tasq {

namespace {

__device__ __forceinline__ float finish_value(const LayerDesc &d, int m, int n, int32_t s,
                                              float zoff)
{
    float scale, corr = 0.0f, bias = 0.0f, extra = 0.0f;
    if (d.act) {
        scale = d.act[0] * d.sw[n];
        corr = (128.0f - d.act[1]) * (float)d.colsums[(d.bits - 1) * d.N + n];
    } else {
        scale = d.sx * d.sw[n];
    }
    if (d.bias)
        bias = d.bias[n];
    if (d.lr_T) {
        const float *t = d.lr_T + (size_t)m * d.lr_r;
        const uint16_t *u = d.lr_U + (size_t)n * d.lr_r;
        for (int q = 0; q < d.lr_r; ++q)
            extra = fmaf(t[q], __uint_as_float((uint32_t)u[q] << 16), extra);
    }
    if (d.wz)
        extra += (128.0f - d.wz[n]) * scale * ((float)d.xrs[m] + zoff);
    return ((float)s + corr) * scale + bias + extra;
}

// vec: N % 4 == 0 and 16-byte aligned outputs; four consecutive outputs of
// one row per thread.
__global__ void __launch_bounds__(256) k_split_finish(LayerDesc d, const int32_t *__restrict__ part,
                                                      int splits, bool vec)
{
    const long long MN = (long long)d.M * d.N;
    const long long stride = (long long)gridDim.x * blockDim.x;
    const float zoff = d.act ? (float)d.K * (128.0f - d.act[1]) : 0.0f;
    if (vec) {
        const long long MN4 = MN >> 2;
        const int4 *p4 = reinterpret_cast<const int4 *>(part);
        for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < MN4;
             i += stride) {
            int4 s = p4[i];
            for (int sp = 1; sp < splits; ++sp) {
                const int4 v = p4[sp * MN4 + i];
                s.x += v.x;
                s.y += v.y;
                s.z += v.z;
                s.w += v.w;
            }
            if (d.acc)
                reinterpret_cast<int4 *>(d.acc)[i] = s;
            if (!d.y)
                continue;
            const long long e = i << 2;
            const int m = (int)(e / d.N), n = (int)(e - (long long)m * d.N);
            reinterpret_cast<float4 *>(d.y)[i] =
                make_float4(finish_value(d, m, n, s.x, zoff), finish_value(d, m, n + 1, s.y, zoff),
                            finish_value(d, m, n + 2, s.z, zoff),
                            finish_value(d, m, n + 3, s.w, zoff));
        }
        return;
    }
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < MN; i += stride) {
        int32_t s = 0;
        for (int sp = 0; sp < splits; ++sp)
            s += part[sp * MN + i];
        if (d.acc)
            d.acc[i] = s;
        if (!d.y)
            continue;
        const int m = (int)(i / d.N), n = (int)(i - (long long)m * d.N);
        d.y[i] = finish_value(d, m, n, s, zoff);
    }
}

}  // namespace

hipError_t launch_split_finish(const LayerDesc &d, const int32_t *part, int splits,
                               hipStream_t stream)
{
    const long long MN = (long long)d.M * d.N;
    const bool vec = (d.N % 4) == 0 && (reinterpret_cast<uintptr_t>(d.acc) & 15) == 0 &&
                     (reinterpret_cast<uintptr_t>(d.y) & 15) == 0;
    long long g = ((vec ? MN / 4 : MN) + 255) / 256;
    if (g > 8192)
        g = 8192;
    hipLaunchKernelGGL(k_split_finish, dim3((unsigned)(g < 1 ? 1 : g)), dim3(256), 0, stream, d,
                       part, splits, vec);
    return hipGetLastError();
}

}  // namespace tasq
