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
// share of the codes.  No atomics and no buffer to clear beforehand.  The
// batched form runs the passes of many tensors in few launches.
#include <vector>

#include "tasq_internal.h"

namespace tasq {

namespace {

// Order-preserving map of a finite float to uint32, so that min / max are
// unsigned integer min / max, whatever order the partial ranges are folded in.
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

// Per-workgroup range of x as order keys: workgroup g of G writes its
// minimum key to part[2g] and its maximum key to part[2g + 1] (no atomics:
// the quantizer folds the partial ranges).  The first 4*n4 elements are read
// as float4 (n4 = 0 when x is not 16-byte aligned), four loads in flight per
// thread.
__device__ __forceinline__ void act_range(const float *__restrict__ x, long long n, long long n4,
                                          uint32_t *__restrict__ part, int g, int G)
{
    __shared__ uint32_t smin[4], smax[4];
    float mn = __builtin_huge_valf(), mx = -__builtin_huge_valf();
    const long long stride = (long long)G * blockDim.x;
    const float4 *x4 = reinterpret_cast<const float4 *>(x);
    long long i = (long long)g * blockDim.x + threadIdx.x;
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
    for (long long t = (n4 << 2) + (long long)g * blockDim.x + threadIdx.x; t < n; t += stride) {
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
        part[2 * g] = kmn;
        part[2 * g + 1] = kmx;
    }
}

__global__ void __launch_bounds__(256) k_act_range(const float *__restrict__ x, long long n,
                                                   long long n4, uint32_t *__restrict__ part)
{
    act_range(x, n, n4, part, blockIdx.x, gridDim.x);
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

// Every workgroup (g of Q) folds the G partial ranges (a few KB, cache
// resident) into alpha and z, then writes the codes of its share; workgroup
// 0 also publishes alpha and z.  n4 as in act_range, with q 4-byte aligned
// whenever n4 > 0.
__device__ __forceinline__ void act_quantize(const float *__restrict__ x, long long n,
                                             long long n4, int8_t *__restrict__ q, float *params,
                                             int G, int g, int Q)
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
    if (g == 0 && threadIdx.x == 0) {
        params[0] = alpha;
        params[1] = z;
    }
    const long long stride = (long long)Q * blockDim.x;
    const float4 *x4 = reinterpret_cast<const float4 *>(x);
    char4 *q4 = reinterpret_cast<char4 *>(q);
    long long i = (long long)g * blockDim.x + threadIdx.x;
    for (; i + 3 * stride < n4; i += 4 * stride) {
        float4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            v[u] = x4[i + u * stride];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            q4[i + u * stride] = make_char4(code_of(v[u].x, alpha, z), code_of(v[u].y, alpha, z),
                                            code_of(v[u].z, alpha, z), code_of(v[u].w, alpha, z));
    }
    for (; i < n4; i += stride) {
        const float4 v = x4[i];
        q4[i] = make_char4(code_of(v.x, alpha, z), code_of(v.y, alpha, z), code_of(v.z, alpha, z),
                           code_of(v.w, alpha, z));
    }
    for (long long i = (n4 << 2) + (long long)g * blockDim.x + threadIdx.x; i < n; i += stride)
        q[i] = code_of(x[i], alpha, z);
}

__global__ void __launch_bounds__(256) k_act_quantize(const float *__restrict__ x, long long n,
                                                      long long n4, int8_t *__restrict__ q,
                                                      float *params, int G)
{
    act_quantize(x, n, n4, q, params, G, blockIdx.x, gridDim.x);
}

// Many tensors in one launch: each task is one tensor's range pass or its
// code pass, run by a contiguous run of the launch's workgroups exactly as
// the single-tensor kernels run it, so the codes and scales are those of the
// single-tensor calls.  The task list travels in the kernel arguments.
struct ActTask {
    const float *x;
    int8_t *q;
    float *params;
    long long n, n4;
    int first;      // first workgroup of the task in the launch
    int wgs;        // its workgroups
    int parts;      // workgroups (partial ranges) of the tensor's range pass
    int quant;      // 0: range pass, 1: code pass
};
constexpr int kActBatchTasks = 16;
struct ActLaunch {
    ActTask t[kActBatchTasks];
    int ntasks;
};

__global__ void __launch_bounds__(256) k_act_batch(const ActLaunch L)
{
    int i = 0;
    while (i + 1 < L.ntasks && (int)blockIdx.x >= L.t[i + 1].first)
        ++i;
    const ActTask &t = L.t[i];
    const int g = (int)blockIdx.x - t.first;
    if (t.quant)
        act_quantize(t.x, t.n, t.n4, t.q, t.params, t.parts, g, t.wgs);
    else
        act_range(t.x, t.n, t.n4, reinterpret_cast<uint32_t *>(t.params + kActHeader), g,
                  t.parts);
}

// ------------------------------------------------- low-rank down projection
//
// T = x~ D^T for the 16-bit low-rank branch: x~ is x rounded to bfloat16
// (nearest, ties to even), D [r x K] bfloat16, T fp32 [M x r], r <= 32.
// One workgroup per 32-row block (grid-stride over blocks); its 8 waves take
// interleaved 16-wide K steps, each a v_mfma_f32_32x32x16_bf16 with lane l
// feeding row l%32 of x and column l%32 of D^T (columns past r are zero).
// The waves' partial blocks are summed through LDS in a fixed order, so T
// does not depend on timing.  The same pass can fold the range of x (one
// partial per workgroup, as k_act_range), so that quantizing the codes and
// projecting share one read of x.

typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));

constexpr int kDownWaves = 16;

__device__ __forceinline__ uint32_t bf16_rne(float f)
{
    const uint32_t u = __float_as_uint(f);
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ v4u pack_bf16(float4 lo, float4 hi)
{
    return v4u{bf16_rne(lo.x) | (bf16_rne(lo.y) << 16), bf16_rne(lo.z) | (bf16_rne(lo.w) << 16),
               bf16_rne(hi.x) | (bf16_rne(hi.y) << 16), bf16_rne(hi.z) | (bf16_rne(hi.w) << 16)};
}

__device__ __forceinline__ void fold_range(float4 v, float &mn, float &mx)
{
    mn = fminf(fminf(mn, v.x), fminf(v.y, fminf(v.z, v.w)));
    mx = fmaxf(fmaxf(mx, v.x), fmaxf(v.y, fmaxf(v.z, v.w)));
}

// FAST: K % 8 == 0 and x, D 16-byte aligned, so an in-range K step covers
// all 8 elements of a lane; each wave then issues the loads of 4 of its K
// steps before their MFMAs (enough bytes in flight with one workgroup per
// CU).  Otherwise every element is loaded on its own with bounds checks.
template <bool RANGE, bool FAST>
__global__ void __launch_bounds__(64 * kDownWaves)
k_lowrank_down(const float *__restrict__ x, int M, int K, const uint16_t *__restrict__ D, int r,
               float *__restrict__ T, uint32_t *__restrict__ part)
{
    __shared__ float red[kDownWaves][16][64];
    __shared__ uint32_t smin[kDownWaves], smax[kDownWaves];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int half = lane >> 5;
    const int j = lane & 31;                         // column of D^T this lane feeds
    const int nsteps = (K + 15) / 16;
    const int nblocks = (M + 31) / 32;
    float mn = __builtin_huge_valf(), mx = -__builtin_huge_valf();

    for (int rb = blockIdx.x; rb < nblocks; rb += gridDim.x) {
        const int row = rb * 32 + j;
        const bool rok = row < M;
        const float *xr = x + (size_t)(rok ? row : 0) * (size_t)K;
        const uint16_t *dr = D + (size_t)(j < r ? j : 0) * (size_t)K;
        v16f acc = {};
        if constexpr (FAST) {
            constexpr int U = 4;
            for (int s0 = wave; s0 < nsteps; s0 += U * kDownWaves) {
                float4 lo[U], hi[U];
                v4u bw[U];
                bool ok[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int k = 16 * (s0 + u * kDownWaves) + 8 * half;
                    const bool kin = k < K;
                    ok[u] = rok && kin;
                    lo[u] = make_float4(0.f, 0.f, 0.f, 0.f);
                    hi[u] = lo[u];
                    if (ok[u]) {
                        const float4 *p = reinterpret_cast<const float4 *>(xr + k);
                        lo[u] = p[0];
                        hi[u] = p[1];
                    }
                    bw[u] = v4u{0, 0, 0, 0};
                    if (j < r && kin)
                        bw[u] = *reinterpret_cast<const v4u *>(dr + k);
                }
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    if (RANGE && ok[u]) {
                        fold_range(lo[u], mn, mx);
                        fold_range(hi[u], mn, mx);
                    }
                    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(v8bf, pack_bf16(lo[u], hi[u])),
                        __builtin_bit_cast(v8bf, bw[u]), acc, 0, 0, 0);
                }
            }
        } else {
            for (int s = wave; s < nsteps; s += kDownWaves) {
                const int k = 16 * s + 8 * half;
                float xv[8];
                uint32_t dv[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const bool ok = k + e < K;
                    xv[e] = (rok && ok) ? xr[k + e] : 0.f;
                    if (rok && ok) {
                        mn = fminf(mn, xv[e]);
                        mx = fmaxf(mx, xv[e]);
                    }
                    dv[e] = (j < r && ok) ? (uint32_t)dr[k + e] : 0u;
                }
                const v4u bw = v4u{dv[0] | (dv[1] << 16), dv[2] | (dv[3] << 16),
                                   dv[4] | (dv[5] << 16), dv[6] | (dv[7] << 16)};
                const v4u aw = pack_bf16(make_float4(xv[0], xv[1], xv[2], xv[3]),
                                         make_float4(xv[4], xv[5], xv[6], xv[7]));
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, aw),
                                                              __builtin_bit_cast(v8bf, bw), acc,
                                                              0, 0, 0);
            }
        }
        // Register v of lane l is row 8*(v/4) + 4*(l/32) + v%4, column l%32.
#pragma unroll
        for (int v = 0; v < 16; ++v)
            red[wave][v][lane] = acc[v];
        __syncthreads();
        for (int e = threadIdx.x; e < 32 * 32; e += 64 * kDownWaves) {
            const int v = e >> 6, l = e & 63;
            const int orow = rb * 32 + 8 * (v >> 2) + 4 * (l >> 5) + (v & 3);
            const int ocol = l & 31;
            float sum = red[0][v][l];
#pragma unroll
            for (int w = 1; w < kDownWaves; ++w)
                sum += red[w][v][l];
            if (orow < M && ocol < r)
                T[(size_t)orow * (size_t)r + ocol] = sum;
        }
        __syncthreads();
    }
    if (RANGE) {
        uint32_t kmn = order_key(mn), kmx = order_key(mx);
        for (int off = 32; off > 0; off >>= 1) {
            kmn = min(kmn, (uint32_t)__shfl_xor((int)kmn, off));
            kmx = max(kmx, (uint32_t)__shfl_xor((int)kmx, off));
        }
        if (lane == 0) {
            smin[wave] = kmn;
            smax[wave] = kmx;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            for (int w = 1; w < kDownWaves; ++w) {
                kmn = min(kmn, smin[w]);
                kmx = max(kmx, smax[w]);
            }
            part[2 * blockIdx.x] = kmn;
            part[2 * blockIdx.x + 1] = kmx;
        }
    }
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

// Groups of consecutive tensors (at most half a launch's tasks, and about
// 128 MB of x unless a single tensor is larger) run their code pass in the
// launch after their range pass, beside the next group's range pass:
// ceil(n / group) + 1 launches instead of 2 n, and each x is read the second
// time while it is still in the last-level cache.
hipError_t launch_quantize_activations_batch(const ActJob *jobs, int n, hipStream_t stream)
{
    constexpr long long kGroupBytes = 128LL << 20;
    constexpr int kGroupTasks = kActBatchTasks / 2;
    struct Prep {
        ActTask range, quant;
    };
    std::vector<Prep> prep;
    prep.reserve((size_t)n);
    for (int j = 0; j < n; ++j) {
        const ActJob &a = jobs[j];
        const long long cnt = (long long)a.M * a.K;
        if (cnt == 0)
            continue;
        const bool vec = (reinterpret_cast<uintptr_t>(a.x) & 15) == 0 &&
                         (reinterpret_cast<uintptr_t>(a.q) & 3) == 0;
        const long long n4 = vec ? cnt >> 2 : 0;
        const long long items = vec ? (cnt + 3) / 4 : cnt;
        const int G = grid_for(items, 256 * 4, kActPartials);
        ActTask r = {a.x, a.q, a.params, cnt, n4, 0, G, G, 0};
        ActTask q = r;
        q.wgs = grid_for(items, 256, 1024);
        q.quant = 1;
        prep.push_back({r, q});
    }
    // group boundaries
    std::vector<int> bounds{0};
    long long bytes = 0;
    for (int j = 0; j < (int)prep.size(); ++j) {
        const long long b = prep[j].range.n * 4;
        const int in_group = j - bounds.back();
        if (in_group > 0 && (in_group == kGroupTasks || bytes + b > kGroupBytes)) {
            bounds.push_back(j);
            bytes = 0;
        }
        bytes += b;
    }
    bounds.push_back((int)prep.size());
    const int ng = (int)bounds.size() - 1;
    for (int k = 0; k <= ng && !prep.empty(); ++k) {
        ActLaunch L = {};
        int wg = 0;
        auto add = [&](ActTask t) {
            t.first = wg;
            wg += t.wgs;
            L.t[L.ntasks++] = t;
        };
        if (k > 0)
            for (int j = bounds[k - 1]; j < bounds[k]; ++j)
                add(prep[j].quant);
        if (k < ng)
            for (int j = bounds[k]; j < bounds[k + 1]; ++j)
                add(prep[j].range);
        hipLaunchKernelGGL(k_act_batch, dim3(wg), dim3(256), 0, stream, L);
        if (hipError_t e = hipGetLastError(); e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

hipError_t launch_lowrank_down(const float *x, int M, int K, const uint16_t *D, int r, float *T,
                               uint32_t *part, int *groups, hipStream_t stream)
{
    const bool fast = (K % 8) == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0 &&
                      (reinterpret_cast<uintptr_t>(D) & 15) == 0;
    const int G = grid_for(M, 32, kActPartials);
    if (groups)
        *groups = G;
    const dim3 g(G), b(64 * kDownWaves);
    if (part && fast)
        hipLaunchKernelGGL((k_lowrank_down<true, true>), g, b, 0, stream, x, M, K, D, r, T, part);
    else if (part)
        hipLaunchKernelGGL((k_lowrank_down<true, false>), g, b, 0, stream, x, M, K, D, r, T, part);
    else if (fast)
        hipLaunchKernelGGL((k_lowrank_down<false, true>), g, b, 0, stream, x, M, K, D, r, T, part);
    else
        hipLaunchKernelGGL((k_lowrank_down<false, false>), g, b, 0, stream, x, M, K, D, r, T,
                           part);
    return hipGetLastError();
}

hipError_t launch_quantize_activations_lowrank(const float *x, int M, int K, int8_t *q,
                                               float *params, const uint16_t *D, int r, float *T,
                                               hipStream_t stream)
{
    int G = 0;
    uint32_t *part = reinterpret_cast<uint32_t *>(params + kActHeader);
    hipError_t e = launch_lowrank_down(x, M, K, D, r, T, part, &G, stream);
    if (e != hipSuccess)
        return e;
    const long long n = (long long)M * K;
    const bool vec = (reinterpret_cast<uintptr_t>(x) & 15) == 0 &&
                     (reinterpret_cast<uintptr_t>(q) & 3) == 0;
    const long long n4 = vec ? n >> 2 : 0;
    const long long items = vec ? (n + 3) / 4 : n;
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
