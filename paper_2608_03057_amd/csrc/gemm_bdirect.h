// Masked int8 GEMM with the weight operand fed from registers (gfx950).
//
// Same operation as gemm_core.h: acc = X * W_b^T with W_b = W & keep_mask(b)
// (TASQ Sec. 3.2.1 Eq. lsb_masking, App. G.2 Eq. hw_rightshift), int32
// accumulation, fp32 dequant epilogue.
//
// On gfx950 an LDS write of 16 bytes per lane sustains about half the
// bandwidth of an LDS read, and staging both operands through LDS makes the
// LDS, not the MFMA pipe, the bound.  Here only the activation tile is staged
// (shared by the four waves of a block row); each wave loads its weight
// fragments straight into registers with 16-byte buffer loads (the two
// waves sharing a weight slice hit in L1) and applies the mask there.
//
// K order inside a 128-byte K tile: lane half h (= lane / 32) of a 32x32x32
// MFMA takes bytes [64h + 16kk, 64h + 16kk + 16) at sub-step kk, so a lane's
// weight bytes for the whole tile are 64 contiguous bytes; the activation
// fragments are read from LDS with the same permutation.  Any permutation of
// the reduction index applied to both operands leaves the int32 sum unchanged.
//
// Tile: 256x256, 8 waves (2 x 4), wave tile 128x64, BK 128.  Activation K
// tiles go straight from HBM into three LDS stages (buffer_load ... lds, no
// staging registers); registers hold the current and next weight tiles.
// Aligned linear layers only.
#pragma once

#include "gemm_direct.h"

namespace tasq {

struct CfgB {
    static constexpr int BM = 256, BN = 256, BK = 128;
    static constexpr int WAVES_M = 2, WAVES_N = 4, NT = 512, OCC = 2;
    static constexpr int WTM = 128, WTN = 64, FM = 4, FN = 2;
    static constexpr int CPR = BK / 16, KK = BK / 32;
    static constexpr int A_LOADS = BM * CPR / NT;        // direct loads per thread
    static constexpr int SA = BM * CPR;                  // v4i per LDS stage
    static constexpr int NS = 3;                         // LDS stages
    static constexpr int B_LOADS = FN * KK;              // register loads per thread
};

template <class C>
__device__ __forceinline__ void mainloop_bdirect(const LayerDesc &d, uint32_t wmask, int m0,
                                                 int n0, int kb, int ke,
                                                 v16i (&acc)[C::FM][C::FN], v4i *smA)
{
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
    const int h = lane >> 5;

#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
            acc[i][j] = v16i{};

    const int span = ke - kb;
    const int nk = (span + C::BK - 1) / C::BK;
    if (nk <= 0)
        return;
    const int last_valid = span - (nk - 1) * C::BK;
    const bool has_tail = last_valid < C::BK;

    // Activation plan: direct load i of wave w fills LDS chunks
    // (8i + w)*64 + lane of the stage: row chunk / CPR, physical column
    // chunk % CPR holding logical column pc ^ swizzle(row).
    const rsrc_t rX = make_rsrc(d.X, (uint32_t)d.M * (uint32_t)d.K);
    uint32_t offA[C::A_LOADS];
#pragma unroll
    for (int i = 0; i < C::A_LOADS; ++i) {
        const int chunk = (8 * i + wave) * 64 + lane;
        const int r = chunk / C::CPR, pc = chunk % C::CPR;
        const int c = swz<C::CPR>(r, pc);
        const int m = m0 + r;
        offA[i] = m < d.M ? (uint32_t)m * (uint32_t)d.K + (uint32_t)(kb + 16 * c) : kOOB;
    }
    // weight fragments: lane half h of column n reads bytes 64h .. 64h+63
    const rsrc_t rW = make_rsrc(d.W, (uint32_t)d.N * (uint32_t)d.K);
    uint32_t offB[C::FN];
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
        const int n = n0 + wn * C::WTN + j * 32 + (lane & 31);
        offB[j] = n < d.N ? (uint32_t)n * (uint32_t)d.K + (uint32_t)(kb + 64 * h) : kOOB;
    }

    v4i vb[2][C::FN][C::KK];
    char *smc = reinterpret_cast<char *>(smA);
    auto issueA = [&](int t, int stage) {
        char *base = smc + stage * C::SA * 16;
#pragma unroll
        for (int i = 0; i < C::A_LOADS; ++i)
            ld_lds16(rX, base + (8 * i + wave) * 1024, offA[i] + (uint32_t)t * C::BK);
    };
    auto loadB = [&](int t, v4i (&b)[C::FN][C::KK]) {
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
#pragma unroll
            for (int kk = 0; kk < C::KK; ++kk)
                b[j][kk] = ld16(rW, offB[j] + (uint32_t)t * C::BK + 16 * kk);
    };

    const int msk = (int)wmask;
    v4i fa[2][C::FM];
    auto readA = [&](int stage, int kk, v4i (&a)[C::FM]) {
        const v4i *A = smA + stage * C::SA;
        const int c = 4 * h + kk;
#pragma unroll
        for (int i = 0; i < C::FM; ++i) {
            const int r = wm * C::WTM + i * 32 + (lane & 31);
            a[i] = A[r * C::CPR + swz<C::CPR>(r, c)];
        }
    };
    // One K tile: A fragments from LDS `stage`, weights from `b`; with
    // `tail`, weight bytes at or past column last_valid read as zero.
    auto compute = [&](int stage, v4i (&b)[C::FN][C::KK], bool tail) {
        readA(stage, 0, fa[0]);
        __builtin_amdgcn_sched_group_barrier(0x100, C::FM, 0);
#pragma unroll
        for (int kk = 0; kk < C::KK; ++kk) {
            if (kk + 1 < C::KK)
                readA(stage, kk + 1, fa[(kk + 1) & 1]);
            v4i bf[C::FN];
#pragma unroll
            for (int j = 0; j < C::FN; ++j) {
                v4i v = b[j][kk];
                v.x &= msk;
                v.y &= msk;
                v.z &= msk;
                v.w &= msk;
                if (tail && 64 * h + 16 * kk >= last_valid)
                    v = zero4();
                bf[j] = v;
            }
#pragma unroll
            for (int i = 0; i < C::FM; ++i)
#pragma unroll
                for (int j = 0; j < C::FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[kk & 1][i], bf[j],
                                                                      acc[i][j], 0, 0, 0);
            if (kk + 1 < C::KK)
                __builtin_amdgcn_sched_group_barrier(0x100, C::FM, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, C::FM * C::FN, 0);
        }
    };

    // Prologue: activation tiles 0 and 1 in flight to LDS stages 0 and 1,
    // weight tile 0 to vb[0]; wait for activation tile 0.
    issueA(0, 0);
    if (nk > 1)
        issueA(1, 1);
    loadB(0, vb[0]);
    if (nk > 1)
        wait_vmcnt<C::A_LOADS + C::B_LOADS>();
    else
        wait_vmcnt<C::B_LOADS>();
    __syncthreads();

    // Tile t: activations in LDS stage t % 3, weights in vb[t & 1].  Issue
    // order per tile: activations of t+2, weights of t+1, then the MFMAs of
    // t; before the barrier, wait until only those two groups may remain in
    // flight, i.e. activation tile t+1 has landed.  The loop is unrolled by
    // two so that the weight registers are indexed statically.
    int stage = 0;
    for (int t0 = 0; t0 < nk; t0 += 2) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int t = t0 + u;
            if (t < nk) {
                const int s1 = stage == 2 ? 0 : stage + 1;
                const int s2 = s1 == 2 ? 0 : s1 + 1;
                if (t + 2 < nk)
                    issueA(t + 2, s2);
                if (t + 1 < nk)
                    loadB(t + 1, vb[u ^ 1]);
                compute(stage, vb[u], t + 1 == nk && has_tail);
                if (t + 1 < nk) {
                    if (t + 2 < nk)
                        wait_vmcnt<C::A_LOADS + C::B_LOADS>();
                    else
                        wait_vmcnt<C::B_LOADS>();
                    __syncthreads();
                }
                stage = s1;
            }
        }
    }
}

template <class C>
__global__ void __launch_bounds__(C::NT, C::OCC) k_gemm_bdirect(LayerDesc d)
{
    __shared__ v4i smA[C::NS * C::SA];
    int tm, tn;
    tile_coords(xcd_remap(blockIdx.x, gridDim.x), d.tiles_m, d.tiles_n, tm, tn);
    const int m0 = tm * C::BM, n0 = tn * C::BN;
    v16i acc[C::FM][C::FN];
    mainloop_bdirect<C>(d, keep_mask_dword(d.bits), m0, n0, 0, d.K, acc, smA);
    epilogue<C>(d, m0, n0, acc);
}

// Grouped step over linear layers (see k_masked_gemm_grouped).
template <class C>
__global__ void __launch_bounds__(C::NT, C::OCC)
k_gemm_bdirect_grouped(const LayerDesc *__restrict__ descs, int L, const uint8_t *table, int S,
                       int stage)
{
    __shared__ v4i smA[C::NS * C::SA];
    const int t = xcd_remap(blockIdx.x, gridDim.x);
    int lo = 0, hi = L - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (descs[mid].tile_begin <= t)
            lo = mid;
        else
            hi = mid - 1;
    }
    const LayerDesc d = descs[lo];
    const uint32_t wmask = keep_mask_dword(table[lo * S + stage]);
    int tm, tn;
    tile_coords(t - d.tile_begin, d.tiles_m, d.tiles_n, tm, tn);
    const int m0 = tm * C::BM, n0 = tn * C::BN;
    v16i acc[C::FM][C::FN];
    mainloop_bdirect<C>(d, wmask, m0, n0, 0, d.K, acc, smA);
    epilogue<C>(d, m0, n0, acc);
}

template <class C>
hipError_t launch_bdirect_single(const LayerDesc &din, bool aligned, hipStream_t stream)
{
    LayerDesc d = din;
    fill_tiles<C>(d);
    const long long grid = (long long)d.tiles_m * d.tiles_n;
    if (grid > 0x7fffffffLL || !aligned || d.kind != KIND_LINEAR)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_gemm_bdirect<C>), dim3((unsigned)grid), dim3(C::NT), 0, stream, d);
    return hipGetLastError();
}

template <class C>
hipError_t launch_bdirect_grouped(const LayerDesc *d_descs, int L, int total_tiles,
                                  const uint8_t *d_table, int S, int stage, hipStream_t stream)
{
    hipLaunchKernelGGL((k_gemm_bdirect_grouped<C>), dim3((unsigned)total_tiles), dim3(C::NT), 0,
                       stream, d_descs, L, d_table, S, stage);
    return hipGetLastError();
}

#define TASQ_DEFINE_BDIRECT_TILE(NAME, CFG)                                                   \
    const TileOps &NAME()                                                                     \
    {                                                                                         \
        static const TileOps ops = {{CFG::BM, CFG::BN, CFG::BK}, &launch_bdirect_single<CFG>, \
                                    nullptr, &launch_bdirect_grouped<CFG>, true};             \
        return ops;                                                                           \
    }

}  // namespace tasq
