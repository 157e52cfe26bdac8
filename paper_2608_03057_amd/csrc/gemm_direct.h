// Masked int8 GEMM, direct-to-LDS variant for gfx950.
//
// Same operation as gemm_core.h (acc = X * W_b^T, W_b = W & keep_mask(b),
// fp32 dequant epilogue), organised to cut LDS traffic per MFMA:
//   * 256x256 block tile, 4 waves (2 x 2), each owning a 128x128 tile of
//     v_mfma_i32_32x32x32_i8 accumulators (256 int32 per lane, held in the
//     accumulator registers; one wave per SIMD).  Operand reads fall to
//     8 ds_read_b128 per 16 MFMAs, against 6 per 8 for 128x64 wave tiles.
//   * Global loads go straight into LDS (buffer_load_dwordx4 ... lds: lane l
//     of an instruction writes 16 bytes at M0 + 16*l), so staging needs no
//     registers and no ds_write.  The XOR swizzle of the LDS rows is realised
//     by choosing which global chunk each lane fetches.  Rows past M or N
//     carry an offset past the buffer end and land as zeros.
//   * The LSB mask (TASQ Sec. 3.2.1 Eq. lsb_masking, App. G.2 Eq.
//     hw_rightshift) is applied to the weight fragments after their LDS read:
//     four v_and_b32 per 16 weight bytes a lane feeds to the MFMAs.
//   * NSTAGE K tiles live in LDS; the loads of tile t+NSTAGE-1 are issued
//     while tile t is computed.  One barrier per K tile, placed before the
//     last 32-wide sub-step, so the first fragments of tile t+1 are read
//     while that sub-step's MFMAs run.
// Linear layers with K % 16 == 0 and 16-byte aligned operands only; other
// layers use the staged kernels of gemm_core.h.
#pragma once

#include "gemm_core.h"

namespace tasq {

template <int BK_, int NS_, int WAVES_N_ = 2>
struct CfgD {
    static constexpr int BM = 256, BN = 256, BK = BK_;
    static constexpr int WAVES_M = 2, WAVES_N = WAVES_N_, NWAVES = WAVES_M * WAVES_N;
    static constexpr int NT = NWAVES * 64;
    static constexpr int OCC = NWAVES / 4;               // waves per SIMD
    static constexpr int WTM = 128, WTN = BN / WAVES_N, FM = 4, FN = WTN / 32;
    static constexpr int CPR = BK / 16;                  // 16-byte chunks per row
    static constexpr int NSTAGE = NS_;
    static constexpr int LOADS = BM * CPR / NT;          // per operand per thread
    static constexpr int A_BYTES = BM * BK, STAGE_BYTES = (BM + BN) * BK;
    static constexpr int KK = BK / 32;
    static_assert(CPR == 4 || CPR == 8, "BK must be 64 or 128");
    static_assert(KK % 2 == 0, "an even number of 32-wide sub-steps per K tile");
    static_assert(NSTAGE >= 2 && NSTAGE * STAGE_BYTES <= 160 * 1024, "LDS capacity");
};

typedef __attribute__((address_space(3))) void lds_void_t;

__device__ __forceinline__ void ld_lds16(rsrc_t r, char *lds, uint32_t voff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t *)lds, 16, voff, 0, 0, 0);
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt[3:0] in bits 3:0 and vmcnt[5:4] in bits 15:14; expcnt and lgkmcnt
// left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

template <class C>
__device__ __forceinline__ void mainloop_direct(const LayerDesc &d, uint32_t wmask, int m0,
                                                int n0, int kb, int ke,
                                                v16i (&acc)[C::FM][C::FN], char *sm)
{
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
    constexpr int NS = C::NSTAGE, KK = C::KK;

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

    // Load plan: instruction i of wave w fills LDS chunks (NWAVES*i + w)*64 + lane,
    // i.e. row r = chunk / CPR, physical column pc = chunk % CPR, which holds
    // the logical column c = pc ^ swizzle(r).
    const rsrc_t rX = make_rsrc(d.X, (uint32_t)d.M * (uint32_t)d.K);
    const rsrc_t rW = make_rsrc(d.W, (uint32_t)d.N * (uint32_t)d.K);
    uint32_t offA[C::LOADS], offB[C::LOADS];
#pragma unroll
    for (int i = 0; i < C::LOADS; ++i) {
        const int chunk = (C::NWAVES * i + wave) * 64 + lane;
        const int r = chunk / C::CPR, pc = chunk % C::CPR;
        const int c = swz<C::CPR>(r, pc);           // the XOR swizzle is an involution
        const int m = m0 + r, n = n0 + r;
        offA[i] = m < d.M ? (uint32_t)m * (uint32_t)d.K + (uint32_t)(kb + 16 * c) : kOOB;
        offB[i] = n < d.N ? (uint32_t)n * (uint32_t)d.K + (uint32_t)(kb + 16 * c) : kOOB;
    }
    auto issue = [&](int t, int s) {
        const uint32_t kt = (uint32_t)t * C::BK;
        char *a = sm + s * C::STAGE_BYTES;
        char *b = a + C::A_BYTES;
#pragma unroll
        for (int i = 0; i < C::LOADS; ++i)
            ld_lds16(rX, a + (C::NWAVES * i + wave) * 1024, offA[i] + kt);
#pragma unroll
        for (int i = 0; i < C::LOADS; ++i)
            ld_lds16(rW, b + (C::NWAVES * i + wave) * 1024, offB[i] + kt);
    };

    const int msk = (int)wmask;
    v4i fa[2][C::FM], fb[2][C::FN];
    // Fragments of sub-step kk of the tile in stage s; weight bytes are
    // masked, and with `tail` zeroed at or past column last_valid.
    auto read = [&](int s, int kk, bool tail, v4i (&a)[C::FM], v4i (&b)[C::FN]) {
        const v4i *A = reinterpret_cast<const v4i *>(sm + s * C::STAGE_BYTES);
        const v4i *B = reinterpret_cast<const v4i *>(sm + s * C::STAGE_BYTES + C::A_BYTES);
        const int c = 2 * kk + (lane >> 5);
#pragma unroll
        for (int i = 0; i < C::FM; ++i) {
            const int r = wm * C::WTM + i * 32 + (lane & 31);
            a[i] = A[r * C::CPR + swz<C::CPR>(r, c)];
        }
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
            const int r = wn * C::WTN + j * 32 + (lane & 31);
            v4i v = B[r * C::CPR + swz<C::CPR>(r, c)];
            v.x &= msk;
            v.y &= msk;
            v.z &= msk;
            v.w &= msk;
            if (tail && 16 * c >= last_valid)
                v = zero4();
            b[j] = v;
        }
    };
    auto mfmas = [&](v4i (&a)[C::FM], v4i (&b)[C::FN]) {
#pragma unroll
        for (int i = 0; i < C::FM; ++i)
#pragma unroll
            for (int j = 0; j < C::FN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[i], b[j], acc[i][j], 0, 0, 0);
    };

    // Prologue: tiles 0 .. NS-2 in flight; wait for tile 0.
#pragma unroll
    for (int p = 0; p < NS - 1; ++p)
        if (p < nk)
            issue(p, p);
    if (nk >= NS - 1)
        wait_vmcnt<(NS - 2) * 2 * C::LOADS>();
    else
        wait_vmcnt<0>();
    __syncthreads();
    read(0, 0, nk == 1 && has_tail, fa[0], fb[0]);

    // Tiles 0 .. nk-2 (straight-line MFMA code; the last tile is peeled so
    // that no accumulator crosses a branch).
    int s = 0;                          // stage of tile t
    for (int t = 0; t + 1 < nk; ++t) {
        if (t + NS - 1 < nk)
            issue(t + NS - 1, s == 0 ? NS - 1 : s - 1);
        // sub-steps 0 .. KK-2: reads of kk+1 in flight under the MFMAs of kk
#pragma unroll
        for (int kk = 0; kk + 1 < KK; ++kk) {
            read(s, kk + 1, false, fa[(kk + 1) & 1], fb[(kk + 1) & 1]);
            mfmas(fa[kk & 1], fb[kk & 1]);
            __builtin_amdgcn_sched_group_barrier(0x100, C::FM + C::FN, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, C::FM * C::FN, 0);
        }
        // tile t+1 landed (own loads, then everyone's), and every wave is done
        // reading tile t's stage, which the next issue overwrites
        if (t + NS - 1 < nk)
            wait_vmcnt<(NS - 2) * 2 * C::LOADS>();
        else
            wait_vmcnt<0>();
        __syncthreads();
        const int sn = s + 1 == NS ? 0 : s + 1;
        read(sn, 0, t + 2 == nk && has_tail, fa[0], fb[0]);
        mfmas(fa[(KK - 1) & 1], fb[(KK - 1) & 1]);
        __builtin_amdgcn_sched_group_barrier(0x100, C::FM + C::FN, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, C::FM * C::FN, 0);
        s = sn;
    }
    // last tile
#pragma unroll
    for (int kk = 0; kk + 1 < KK; ++kk) {
        read(s, kk + 1, has_tail, fa[(kk + 1) & 1], fb[(kk + 1) & 1]);
        mfmas(fa[kk & 1], fb[kk & 1]);
        __builtin_amdgcn_sched_group_barrier(0x100, C::FM + C::FN, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, C::FM * C::FN, 0);
    }
    mfmas(fa[(KK - 1) & 1], fb[(KK - 1) & 1]);
}

template <class C>
__global__ void __launch_bounds__(C::NT, C::OCC) k_gemm_direct(LayerDesc d)
{
    __shared__ __attribute__((aligned(16))) char sm[C::NSTAGE * C::STAGE_BYTES];
    int tm, tn;
    tile_coords(xcd_remap(blockIdx.x, gridDim.x), d.tiles_m, d.tiles_n, tm, tn);
    const int m0 = tm * C::BM, n0 = tn * C::BN;
    v16i acc[C::FM][C::FN];
    mainloop_direct<C>(d, keep_mask_dword(d.bits), m0, n0, 0, d.K, acc, sm);
    epilogue<C>(d, m0, n0, acc);
}

// Grouped step over linear layers (see k_masked_gemm_grouped).
template <class C>
__global__ void __launch_bounds__(C::NT, C::OCC)
k_gemm_direct_grouped(const LayerDesc *__restrict__ descs, int L, const uint8_t *table, int S,
                      int stage)
{
    __shared__ __attribute__((aligned(16))) char sm[C::NSTAGE * C::STAGE_BYTES];
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
    mainloop_direct<C>(d, wmask, m0, n0, 0, d.K, acc, sm);
    epilogue<C>(d, m0, n0, acc);
}

template <class C>
hipError_t launch_direct_single(const LayerDesc &din, bool aligned, hipStream_t stream)
{
    LayerDesc d = din;
    fill_tiles<C>(d);
    const long long grid = (long long)d.tiles_m * d.tiles_n;
    if (grid > 0x7fffffffLL)
        return hipErrorInvalidValue;
    if (!aligned || d.kind != KIND_LINEAR)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_gemm_direct<C>), dim3((unsigned)grid), dim3(C::NT), 0, stream, d);
    return hipGetLastError();
}

template <class C>
hipError_t launch_direct_grouped(const LayerDesc *d_descs, int L, int total_tiles,
                                 const uint8_t *d_table, int S, int stage, hipStream_t stream)
{
    hipLaunchKernelGGL((k_gemm_direct_grouped<C>), dim3((unsigned)total_tiles), dim3(C::NT), 0,
                       stream, d_descs, L, d_table, S, stage);
    return hipGetLastError();
}

// Dispatch entry of a direct-to-LDS configuration: linear, aligned layers
// only (TileOps::linear_only); the bit-plane path is not provided.
#define TASQ_DEFINE_DIRECT_TILE(NAME, CFG)                                                   \
    const TileOps &NAME()                                                                    \
    {                                                                                        \
        static const TileOps ops = {{CFG::BM, CFG::BN, CFG::BK}, &launch_direct_single<CFG>, \
                                    nullptr, &launch_direct_grouped<CFG>, true};             \
        return ops;                                                                          \
    }

}  // namespace tasq
