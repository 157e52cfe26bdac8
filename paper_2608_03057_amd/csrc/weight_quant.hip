// Offline weight quantizer (App. A.1.1, Eqs. weight_quant, weight_scale,
// weight_dequant) at the stored precision n = 8, one scale and zero point
// per output channel:
//
//   alpha = (max(w) - min(w)) / 256,  z = -min(w) / alpha  (z kept real),
//   Q = clamp(floor(w / alpha + z), 0, 255),   stored as the code Q - 128,
//   w_hat = 256/255 * alpha * (Q - z) = sw * (Q - z),  sw = alpha * 256 / 255.
//
// The 2^n grid makes the lower-precision codes prefixes of the stored one
// (Eq. truncquant), so the LSB mask of the GEMM applies to these codes as
// they are.  Decisions are taken in IEEE single precision in the order
// written (correctly rounded division, then addition, then floor); a
// constant row takes alpha = 1, z = -min.
//
// Also the row sums of int8 activation codes, which the weight zero point
// needs: sum_k x_hat w_hat_b = sw (sum_k x_hat W_b + (128 - z) sum_k x_hat).
#include "tasq.h"
#include "tasq_internal.h"

#include <algorithm>
#include <vector>

namespace tasq {

namespace {

// fp32 code decision of value v (the order written in the header comment).
__device__ __forceinline__ int8_t weight_code(float v, float alpha, float z)
{
    float f = floorf(__fadd_rn(__fdiv_rn(v, alpha), z));
    f = fminf(fmaxf(f, 0.0f), 255.0f);
    return (int8_t)((int)f - 128);
}

__device__ __forceinline__ void range_to_scale(float mn, float mx, float &alpha, float &z)
{
    if (mx == mn) {
        alpha = 1.0f;
        z = -mn;
    } else {
        alpha = __fdiv_rn(mx - mn, 256.0f);
        z = __fdiv_rn(-mn, alpha);
    }
}

// Output channel n of one weight, by one wave: range, then codes (the row
// read a second time, from L2); lane 0 writes the channel's alpha, z and
// sw.  vec: W rows 16-byte aligned (K % 4 == 0 and W aligned) and Q rows
// 4-byte aligned.
__device__ __forceinline__ void quantize_row(const float *__restrict__ W, int K,
                                             int8_t *__restrict__ Q, float *__restrict__ alpha_out,
                                             float *__restrict__ z_out,
                                             float *__restrict__ sw_out, bool vec, long long n)
{
    const int lane = threadIdx.x & 63;
    const float *w = W + n * (long long)K;
    int8_t *q = Q + n * (long long)K;
    float mn = __builtin_huge_valf(), mx = -__builtin_huge_valf();
    const int K4 = vec ? K / 4 : 0;
    const float4 *w4 = reinterpret_cast<const float4 *>(w);
    for (int i = lane; i < K4; i += 64) {
        const float4 v = w4[i];
        mn = fminf(fminf(mn, v.x), fminf(v.y, fminf(v.z, v.w)));
        mx = fmaxf(fmaxf(mx, v.x), fmaxf(v.y, fmaxf(v.z, v.w)));
    }
    for (int k = 4 * K4 + lane; k < K; k += 64) {
        mn = fminf(mn, w[k]);
        mx = fmaxf(mx, w[k]);
    }
    for (int off = 32; off > 0; off >>= 1) {
        mn = fminf(mn, __shfl_xor(mn, off));
        mx = fmaxf(mx, __shfl_xor(mx, off));
    }
    float alpha, z;
    range_to_scale(mn, mx, alpha, z);
    auto code = [&](float v) -> int8_t { return weight_code(v, alpha, z); };
    char4 *q4 = reinterpret_cast<char4 *>(q);
    for (int i = lane; i < K4; i += 64) {
        const float4 v = w4[i];
        q4[i] = make_char4(code(v.x), code(v.y), code(v.z), code(v.w));
    }
    for (int k = 4 * K4 + lane; k < K; k += 64)
        q[k] = code(w[k]);
    if (lane == 0) {
        alpha_out[n] = alpha;
        z_out[n] = z;
        sw_out[n] = __fdiv_rn(alpha * 256.0f, 255.0f);
    }
}

// One wave per output channel of one weight.
__global__ void __launch_bounds__(256) k_weight_quantize(const float *__restrict__ W, int N, int K,
                                                         int8_t *__restrict__ Q,
                                                         float *__restrict__ alpha_out,
                                                         float *__restrict__ z_out,
                                                         float *__restrict__ sw_out, bool vec)
{
    const long long n = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (n >= N)
        return;
    quantize_row(W, K, Q, alpha_out, z_out, sw_out, vec, n);
}

// Up to 16 weights per launch, travelling by value: the launch's rows are
// the weights' rows end to end, one wave per row (first: the task's first
// row in the launch).
struct WeightTask {
    const float *W;
    int8_t *Q;
    float *alpha, *z, *sw;
    long long first;
    int N, K;
    int vec;
};
constexpr int kWeightBatchTasks = 16;
struct WeightLaunch {
    WeightTask t[kWeightBatchTasks];
    int ntasks;
};

__global__ void __launch_bounds__(256) k_weight_quantize_batch(WeightLaunch L)
{
    const long long g = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
    int j = 0;
    while (j + 1 < L.ntasks && g >= L.t[j + 1].first)
        ++j;
    const WeightTask &t = L.t[j];
    const long long n = g - t.first;
    if (n < 0 || n >= t.N)
        return;
    quantize_row(t.W, t.K, t.Q, t.alpha, t.z, t.sw, t.vec != 0, n);
}

// One wave per row: sum_k X[m][k] of int8 codes, exact in int32 for
// K <= 2^24.
__global__ void __launch_bounds__(256) k_row_sums(const int8_t *__restrict__ X, int M, int K,
                                                  int32_t *__restrict__ out, bool vec)
{
    const int lane = threadIdx.x & 63;
    const long long m = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (m >= M)
        return;
    const int8_t *x = X + m * (long long)K;
    int s = 0;
    const int K4 = vec ? K / 4 : 0;
    const char4 *x4 = reinterpret_cast<const char4 *>(x);
    for (int i = lane; i < K4; i += 64) {
        const char4 v = x4[i];
        s += (int)v.x + (int)v.y + (int)v.z + (int)v.w;
    }
    for (int k = 4 * K4 + lane; k < K; k += 64)
        s += x[k];
    for (int off = 32; off > 0; off >>= 1)
        s += __shfl_xor(s, off);
    if (lane == 0)
        out[m] = s;
}

}  // namespace

hipError_t launch_quantize_weights(const float *W, int N, int K, int8_t *Q, float *alpha,
                                   float *z, float *sw, hipStream_t stream)
{
    const bool vec = (K % 4) == 0 && (reinterpret_cast<uintptr_t>(W) & 15) == 0 &&
                     (reinterpret_cast<uintptr_t>(Q) & 3) == 0;
    hipLaunchKernelGGL(k_weight_quantize, dim3((unsigned)((N + 3) / 4)), dim3(256), 0, stream, W,
                       N, K, Q, alpha, z, sw, vec);
    return hipGetLastError();
}

// Weights of the batch, up to 16 per launch (validated by the caller).
hipError_t launch_quantize_weights_batch(const tasq_weight_job *jobs, int n, hipStream_t stream)
{
    WeightLaunch L = {};
    long long rows = 0;
    auto flush = [&]() -> hipError_t {
        if (L.ntasks == 0)
            return hipSuccess;
        hipLaunchKernelGGL(k_weight_quantize_batch, dim3((unsigned)((rows + 3) / 4)), dim3(256),
                           0, stream, L);
        L = {};
        rows = 0;
        return hipGetLastError();
    };
    for (int j = 0; j < n; ++j) {
        const tasq_weight_job &a = jobs[j];
        if (a.N == 0)
            continue;
        // a launch's grid stays below 2^30 workgroups of 4 rows
        if (rows + a.N > (1LL << 32))
            if (hipError_t e = flush(); e != hipSuccess)
                return e;
        const bool vec = (a.K % 4) == 0 && (reinterpret_cast<uintptr_t>(a.W) & 15) == 0 &&
                         (reinterpret_cast<uintptr_t>(a.W_out) & 3) == 0;
        L.t[L.ntasks++] = {a.W, a.W_out, a.alpha_out, a.z_out, a.sw_out, rows, a.N, a.K,
                           vec ? 1 : 0};
        rows += a.N;
        if (L.ntasks == kWeightBatchTasks)
            if (hipError_t e = flush(); e != hipSuccess)
                return e;
    }
    return flush();
}

hipError_t launch_row_sums(const int8_t *X, int M, int K, int32_t *out, hipStream_t stream)
{
    const bool vec = (K % 4) == 0 && (reinterpret_cast<uintptr_t>(X) & 3) == 0;
    hipLaunchKernelGGL(k_row_sums, dim3((unsigned)((M + 3) / 4)), dim3(256), 0, stream, X, M, K,
                       out, vec);
    return hipGetLastError();
}

}  // namespace tasq

// The batched offline weight quantizer: every job validated as
// tasq_quantize_weights validates its arguments, before any launch.
extern "C" int tasq_quantize_weights_batch(const tasq_weight_job *jobs, int n, void *stream)
{
    if (n < 0)
        return TASQ_ERR_RANGE;
    if (n == 0)
        return TASQ_OK;
    if (!jobs)
        return TASQ_ERR_NULL;
    std::vector<const float *> bufs;
    bufs.reserve((size_t)n);
    for (int j = 0; j < n; ++j) {
        const tasq_weight_job &a = jobs[j];
        if (a.N < 0 || a.K < 0 || (a.N > 0 && a.K == 0))
            return TASQ_ERR_DIM;
        if (a.K > TASQ_MAX_K)
            return TASQ_ERR_OVERFLOW;
        if (a.N == 0)
            continue;
        if (!a.W || !a.W_out || !a.alpha_out || !a.z_out || !a.sw_out)
            return TASQ_ERR_NULL;
        if ((reinterpret_cast<uintptr_t>(a.W) & 3) || (reinterpret_cast<uintptr_t>(a.alpha_out) & 3) ||
            (reinterpret_cast<uintptr_t>(a.z_out) & 3) || (reinterpret_cast<uintptr_t>(a.sw_out) & 3))
            return TASQ_ERR_ALIGN;
        if ((long long)a.N * a.K >= (1LL << 40))
            return TASQ_ERR_DIM;
        bufs.push_back(a.alpha_out);
    }
    std::sort(bufs.begin(), bufs.end());
    if (std::adjacent_find(bufs.begin(), bufs.end()) != bufs.end())
        return TASQ_ERR_RANGE;
    hipError_t e = tasq::launch_quantize_weights_batch(jobs, n, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? TASQ_OK : TASQ_ERR_HIP;
}
