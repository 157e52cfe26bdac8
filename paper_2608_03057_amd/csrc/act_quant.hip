// Asymmetric 8-bit activation quantizer (App. A.1.2, Eqs. act_quant and
// act_scale) feeding the masked GEMM, and the per-precision channel sums of
// the masked weight that its zero point needs.
//
//   alpha = (max(x) - min(x)) / 255,  z = -min(x) / alpha  (per tensor),
//   Q = clamp(round_to_nearest(x / alpha + z), 0, 255),
//   stored as the signed code Q - 128 (int8), the operand of the int8 MFMA.
//
// With x_hat = alpha (Q - z) the layer output is
//   sum_k x_hat_k * sw[n] W_b[n][k] = alpha sw[n] (acc[n] + (128 - z) colsum_b[n]),
//   acc[n] = sum_k (Q_k - 128) W_b[n][k],  colsum_b[n] = sum_k W_b[n][k],
// which the GEMM epilogue evaluates.  The codes are decided in IEEE single
// precision (correctly rounded division, then addition, ties to even);
// when max == min, alpha = 1 and z = -min (every code 0, dequantising to min).
//
// Two launches: per-workgroup ranges into the params buffer's partial slots,
// then a pass in which every workgroup folds those partials and writes its
// share of the codes.  No atomics and no buffer to clear beforehand.
#include "tasq_internal.h"

namespace tasq {

namespace {

// Order-preserving map of a finite float to uint32, so that min / max are
// unsigned integer min / max (atomics on global memory).
__device__ __forceinline__ uint32_t order_key(float f)
{
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float order_value(uint32_t k)
{
    const uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
    return __uint_as_float(u);
}

// Per-workgroup range of x as order keys: workgroup g writes its minimum
// key to part[2g] and its maximum key to part[2g + 1] (no atomics: the
// quantizer folds the partial ranges).  The first 4*n4 elements are read as
// float4 (n4 = 0 when x is not 16-byte aligned), four loads in flight per
// thread.
__global__ void __launch_bounds__(256) k_act_range(const float *__restrict__ x, long long n,
                                                   long long n4, uint32_t *__restrict__ part)
{
    __shared__ uint32_t smin[4], smax[4];
    float mn = __builtin_huge_valf(), mx = -__builtin_huge_valf();
    const long long stride = (long long)gridDim.x * blockDim.x;
    const float4 *x4 = reinterpret_cast<const float4 *>(x);
    long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    for (; i + 3 * stride < n4; i += 4 * stride) {
        float4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            v[u] = x4[i + u * stride];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            mn = fminf(fminf(mn, v[u].x), fminf(v[u].y, fminf(v[u].z, v[u].w)));
            mx = fmaxf(fmaxf(mx, v[u].x), fmaxf(v[u].y, fmaxf(v[u].z, v[u].w)));
        }
    }
    for (; i < n4; i += stride) {
        const float4 v = x4[i];
        mn = fminf(fminf(mn, v.x), fminf(v.y, fminf(v.z, v.w)));
        mx = fmaxf(fmaxf(mx, v.x), fmaxf(v.y, fmaxf(v.z, v.w)));
    }
    for (long long t = (n4 << 2) + (long long)blockIdx.x * blockDim.x + threadIdx.x; t < n;
         t += stride) {
        mn = fminf(mn, x[t]);
        mx = fmaxf(mx, x[t]);
    }
    // Keys order -0 below +0, so the fold below is independent of the order
    // in which the partial ranges meet.
    uint32_t kmn = order_key(mn), kmx = order_key(mx);
    for (int off = 32; off > 0; off >>= 1) {
        kmn = min(kmn, (uint32_t)__shfl_xor((int)kmn, off));
        kmx = max(kmx, (uint32_t)__shfl_xor((int)kmx, off));
    }
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0) {
        smin[wave] = kmn;
        smax[wave] = kmx;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < 4; ++w) {
            kmn = min(kmn, smin[w]);
            kmx = max(kmx, smax[w]);
        }
        part[2 * blockIdx.x] = kmn;
        part[2 * blockIdx.x + 1] = kmx;
    }
}

__device__ __forceinline__ void scale_of(uint32_t kmn, uint32_t kmx, float &alpha, float &z)
{
    const float mn = order_value(kmn), mx = order_value(kmx);
    if (mx == mn) {
        alpha = 1.0f;
        z = -mn;
    } else {
        alpha = __fdiv_rn(mx - mn, 255.0f);
        z = __fdiv_rn(-mn, alpha);
    }
}

__device__ __forceinline__ int8_t code_of(float x, float alpha, float z)
{
    float r = rintf(__fadd_rn(__fdiv_rn(x, alpha), z));
    r = fminf(fmaxf(r, 0.0f), 255.0f);
    return (int8_t)((int)r - 128);
}

// Every workgroup folds the G partial ranges (a few KB, cache resident) into
// alpha and z, then writes the codes of its share; workgroup 0 also
// publishes alpha and z.  n4 as in k_act_range, with q 4-byte aligned
// whenever n4 > 0.
__global__ void __launch_bounds__(256) k_act_quantize(const float *__restrict__ x, long long n,
                                                      long long n4, int8_t *__restrict__ q,
                                                      float *params, int G)
{
    __shared__ uint32_t smin[4], smax[4];
    const uint32_t *part = reinterpret_cast<const uint32_t *>(params + kActHeader);
    uint32_t kmn = 0xffffffffu, kmx = 0u;
    for (int g = threadIdx.x; g < G; g += blockDim.x) {
        kmn = min(kmn, part[2 * g]);
        kmx = max(kmx, part[2 * g + 1]);
    }
    for (int off = 32; off > 0; off >>= 1) {
        kmn = min(kmn, (uint32_t)__shfl_xor((int)kmn, off));
        kmx = max(kmx, (uint32_t)__shfl_xor((int)kmx, off));
    }
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0) {
        smin[wave] = kmn;
        smax[wave] = kmx;
    }
    __syncthreads();
    kmn = min(min(smin[0], smin[1]), min(smin[2], smin[3]));
    kmx = max(max(smax[0], smax[1]), max(smax[2], smax[3]));
    float alpha, z;
    scale_of(kmn, kmx, alpha, z);
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        params[0] = alpha;
        params[1] = z;
    }
    const long long stride = (long long)gridDim.x * blockDim.x;
    const float4 *x4 = reinterpret_cast<const float4 *>(x);
    char4 *q4 = reinterpret_cast<char4 *>(q);
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
        const float4 v = x4[i];
        q4[i] = make_char4(code_of(v.x, alpha, z), code_of(v.y, alpha, z), code_of(v.z, alpha, z),
                           code_of(v.w, alpha, z));
    }
    for (long long i = (n4 << 2) + (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += stride)
        q[i] = code_of(x[i], alpha, z);
}

// One wave per output channel: the eight sums sum_k W_b[n][k], b = 1..8.
__global__ void __launch_bounds__(256) k_weight_colsums(const int8_t *__restrict__ W, int N, int K,
                                                        int32_t *__restrict__ colsums)
{
    const int lane = threadIdx.x & 63;
    const long long n = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (n >= N)
        return;
    const int8_t *row = W + n * (long long)K;
    int s[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int k = lane; k < K; k += 64) {
        const int w = row[k];
#pragma unroll
        for (int b = 1; b <= 8; ++b)
            s[b - 1] += (int)(int8_t)(w & (0xff << (8 - b)));
    }
#pragma unroll
    for (int b = 0; b < 8; ++b)
        for (int off = 32; off > 0; off >>= 1)
            s[b] += __shfl_xor(s[b], off);
    if (lane == 0) {
#pragma unroll
        for (int b = 0; b < 8; ++b)
            colsums[(long long)b * N + n] = s[b];
    }
}

int grid_for(long long items, int per_block, int cap)
{
    long long g = (items + per_block - 1) / per_block;
    if (g > cap)
        g = cap;
    return g < 1 ? 1 : (int)g;
}

}  // namespace

hipError_t launch_quantize_activations(const float *x, long long n, int8_t *q, float *params,
                                       hipStream_t stream)
{
    const bool vec = (reinterpret_cast<uintptr_t>(x) & 15) == 0 &&
                     (reinterpret_cast<uintptr_t>(q) & 3) == 0;
    const long long n4 = vec ? n >> 2 : 0;
    const long long items = vec ? (n + 3) / 4 : n;
    // Range: at most kActPartials workgroups, four float4 per thread per pass.
    const int G = grid_for(items, 256 * 4, kActPartials);
    uint32_t *part = reinterpret_cast<uint32_t *>(params + kActHeader);
    hipLaunchKernelGGL(k_act_range, dim3(G), dim3(256), 0, stream, x, n, n4, part);
    hipLaunchKernelGGL(k_act_quantize, dim3(grid_for(items, 256, 1024)), dim3(256), 0, stream, x,
                       n, n4, q, params, G);
    return hipGetLastError();
}

hipError_t launch_weight_colsums(const int8_t *W, int N, int K, int32_t *colsums,
                                 hipStream_t stream)
{
    hipLaunchKernelGGL(k_weight_colsums, dim3((unsigned)((N + 3) / 4)), dim3(256), 0, stream, W,
                       N, K, colsums);
    return hipGetLastError();
}

}  // namespace tasq
