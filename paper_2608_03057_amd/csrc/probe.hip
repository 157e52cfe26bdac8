// Measurement probe for the benchmark (libtasq_probe.so, not part of the
// TASQ C ABI): the int8 matrix-instruction rate the chip sustains with no
// memory traffic, to set the measured compute ceiling beside the datasheet
// peak.
//
// Every wave issues `iters` rounds of eight independent
// v_mfma_i32_32x32x32_i8 (eight accumulators, so no instruction waits on the
// previous one) on register operands, then folds its accumulators into one
// int32 per lane so that the work cannot be dropped.  The loop count is
// fixed by the caller; no memory is touched until the final store.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kChains = 8;

__global__ void __launch_bounds__(kThreads, 2) k_mfma_peak(int iters, int32_t *sink)
{
    const v4i a = {(int)threadIdx.x, 0x01020304, 0x05060708, 0x090a0b0c};
    const v4i b = {(int)blockIdx.x, 0x0d0e0f10, 0x11121314, 0x15161718};
    v16i acc[kChains];
#pragma unroll
    for (int j = 0; j < kChains; ++j)
        acc[j] = v16i{};
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < kChains; ++j)
            acc[j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc[j], 0, 0, 0);
    }
    int s = 0;
#pragma unroll
    for (int j = 0; j < kChains; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v)
            s += acc[j][v];
    sink[(size_t)blockIdx.x * kThreads + threadIdx.x] = s;
}

}  // namespace

extern "C" {

// Launches `blocks` workgroups of 256 threads, each wave doing iters * 8
// matrix instructions (2 * 32 * 32 * 32 int8 ops each).  sink: device int32
// [blocks * 256], written once per thread.  Returns 0, or -1 for bad
// arguments or a failed launch.
int tasq_probe_mfma_peak(int blocks, int iters, int32_t *sink, void *stream)
{
    if (blocks < 1 || iters < 1 || !sink)
        return -1;
    hipLaunchKernelGGL(k_mfma_peak, dim3((unsigned)blocks), dim3(kThreads), 0,
                       static_cast<hipStream_t>(stream), iters, sink);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

// Matrix instructions per wave-iteration, threads per workgroup: the
// caller's op count is blocks * (256 / 64) * iters * 8 * 65536.
int tasq_probe_mfma_chains(void) { return kChains; }

}  // extern "C"
