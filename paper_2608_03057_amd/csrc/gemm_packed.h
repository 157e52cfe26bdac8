// Masked int8 GEMM with the weight operand streamed from a packed layout
// straight into registers (gfx950).
//
// Same operation as gemm_core.h: acc = X * W_b^T with W_b = W & keep_mask(b)
// (TASQ Sec. 3.2.1 Eq. lsb_masking, App. G.2 Eq. hw_rightshift), int32
// accumulation, fp32 dequant epilogue.  The stored weight buffer is the one
// 8-bit copy shared by every precision, kept in the MFMA operand order
// instead of row-major:
//
//   unit (nb, ks), 1 KB, at byte ((nb * KS + ks) * 64 + l) * 16 holds, for
//   lane l = 0..63, the 16 bytes W[32*nb + l%32][32*ks + 16*(l/32) .. +15];
//   KS = 4 * ceil(K / 128), rows past N and columns past K are zero.
//
// One 16-byte load per lane then fetches one whole 1 KB unit, which is
// exactly a 32x32 B fragment of v_mfma_i32_32x32x32_i8, so the weights need
// no LDS: only the activation tile is staged (two LDS stages), each wave
// loads the fragments of its own output channels one K tile ahead and masks
// them in registers (one v_and_b32 per four weights).  Compared with staging
// both operands, this removes the weight half of the LDS writes and a third
// of the LDS reads, and the activation-only LDS footprint lets the 4-wave
// tiles run two workgroups per CU, so one workgroup's epilogue stores
// overlap the other's MFMAs.
#pragma once

#include "gemm_core.h"

namespace tasq {

template <int BM_, int BN_, int BK_, int WAVES_M_, int WAVES_N_, int OCC_ = 2, int PF_ = 1>
struct CfgP {
    static constexpr int BM = BM_, BN = BN_, BK = BK_;
    static constexpr int WAVES_M = WAVES_M_, WAVES_N = WAVES_N_;
    static constexpr int OCC = OCC_;                    // target waves per SIMD
    static constexpr int NT = WAVES_M * WAVES_N * 64;
    static constexpr int WTM = BM / WAVES_M, WTN = BN / WAVES_N;
    static constexpr int FM = WTM / 32, FN = WTN / 32;
    static constexpr int CPR = BK / 16, KK = BK / 32;
    static constexpr int SA = BM * CPR;                 // v4i per LDS stage
    // LDS of the kernel: two stages, or the epilogue's low-rank operands.
    static constexpr int LR_BYTES = (2 * BM + BN) * kLrPitch + 4 * BM;
    static constexpr int SM = 2 * SA > (LR_BYTES + 15) / 16 ? 2 * SA : (LR_BYTES + 15) / 16;
    static constexpr int A_LOADS = BM * CPR / NT;
    static constexpr int B_LOADS = 0;                   // weights bypass LDS
    static constexpr int PF = PF_;                      // activation K tiles in the ring
    static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile must hold 32x32 blocks");
    static_assert(BK == 64 || BK == 128, "BK must be 64 or 128");
    static_assert((BM * CPR) % NT == 0, "activation loads must divide");
    static_assert(KK % 2 == 0, "an even number of 32-wide sub-steps per K tile");
};

// Bytes of the packed weight buffer of an [N][K] weight.
__host__ __device__ inline size_t packed_weight_bytes(int N, int K)
{
    return (size_t)((N + 31) / 32) * 32 * (size_t)((K + 127) / 128) * 128;
}

// Accumulates all of K for tile (m0, n0).  Schedule as mainloop() in
// gemm_core.h (barrier before the last sub-step, one fragment read after
// each MFMA, PF activation tiles in flight), except that the next
// activation tile is stored half-way through the current one (storing it in
// the sub-step before the barrier measured slower here).
// The weight fragments live in one register buffer per sub-step: as soon as
// the MFMAs of sub-step kk of tile t have taken their (masked) copy, the
// fragment of sub-step kk of tile t+1 is loaded into the same registers, so
// each weight load has one whole K tile to land and only one K tile of
// weights is held in registers.
template <class C, bool ALIGNED, int KIND>
__device__ __forceinline__ void mainloop_packed(const LayerDesc &d, uint32_t wmask, int m0, int n0,
                                                v16i (&acc)[C::FM][C::FN], v4i *sm)
{
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
    constexpr int SA = C::SA, KK = C::KK, PF = C::PF;
    constexpr int WRITE_KK = KK / 2 - 1;

#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
            acc[i][j] = v16i{};
    const int nk = (d.K + C::BK - 1) / C::BK;
    if (nk <= 0)
        return;

    Plan<C, ALIGNED, KIND, false> plan;
    plan.init(d, m0, n0, 0, d.K, tid);
    Regs<C, ALIGNED, KIND, false> ring[PF];

    // This lane's 16 bytes of unit (nb, ks) sit at ((nb*KS + ks)*64 + lane)*16.
    const int KS = (d.K + 127) / 128 * 4;
    const int NB = (d.N + 31) / 32;
    const rsrc_t rW = make_rsrc(d.Wp, (uint32_t)packed_weight_bytes(d.N, d.K));
    uint32_t offB[C::FN];
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
        const int nb = (n0 + wn * C::WTN) / 32 + j;
        offB[j] = nb < NB ? (uint32_t)nb * (uint32_t)KS * 1024u + (uint32_t)lane * 16u : kOOB;
    }
    const int msk = (int)wmask;

    v4i wb[C::FN][KK];
    auto loadB = [&](int t, int kk) {
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
            wb[j][kk] = ld16(rW, offB[j] + (uint32_t)(t * KK + kk) * 1024u);
    };
    v4i fa[2][C::FM];
    auto read = [&](int stage, int kk, v4i (&a)[C::FM]) {
        const v4i *A = sm + stage * SA;
        const int c = 2 * kk + (lane >> 5);
#pragma unroll
        for (int i = 0; i < C::FM; ++i) {
            const int r = wm * C::WTM + i * 32 + (lane & 31);
            a[i] = A[r * C::CPR + swz<C::CPR>(r, c)];
        }
    };
    auto mfmas = [&](v4i (&a)[C::FM], int kk) {
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
            v4i w = wb[j][kk];
            w.x &= msk;
            w.y &= msk;
            w.z &= msk;
            w.w &= msk;
#pragma unroll
            for (int i = 0; i < C::FM; ++i)
                acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[i], w, acc[i][j], 0, 0, 0);
        }
    };

    // Prologue: activation tile 0 into stage 0, tiles 1 .. PF into the ring,
    // weight tile 0 into registers.
    ring[0].load(plan, d, m0, n0, 0, 0u, tid);
    ring[0].store(sm, nullptr, wmask, tid);
#pragma unroll
    for (int u = 0; u < PF; ++u)
        if (1 + u < nk)
            ring[u].load(plan, d, m0, n0, (1 + u) * C::BK, (uint32_t)(1 + u) * C::BK, tid);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
        loadB(0, kk);
    __syncthreads();
    read(0, 0, fa[0]);

    // Tiles 0 .. nk-2; tile t's successor is in ring[t % PF] (the loop is
    // unrolled by PF so that the ring is indexed statically).
    int stage = 0;
    for (int t0 = 0; t0 < nk - 1; t0 += PF) {
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            const int t = t0 + u;
            if (t < nk - 1) {
#pragma unroll
                for (int kk = 0; kk + 1 < KK; ++kk) {
                    read(stage, kk + 1, fa[(kk + 1) & 1]);
                    mfmas(fa[kk & 1], kk);
                    loadB(t + 1, kk);
#pragma unroll
                    for (int i = 0; i < C::FM * C::FN; ++i) {
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                        if (i < C::FM)
                            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    }
                    if (kk == WRITE_KK) {
                        ring[u].store(sm + (stage ^ 1) * SA, nullptr, wmask, tid);
                        if (t + 1 + PF < nk) {
                            const uint32_t off = (uint32_t)(t + 1 + PF) * C::BK;
                            ring[u].load(plan, d, m0, n0, (int)off, off, tid);
                        }
                    }
                }
                __syncthreads();
                read(stage ^ 1, 0, fa[0]);
                mfmas(fa[(KK - 1) & 1], KK - 1);
                loadB(t + 1, KK - 1);
#pragma unroll
                for (int i = 0; i < C::FM * C::FN; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    if (i < C::FM)
                        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                }
                stage ^= 1;
            }
        }
    }
    // Last K tile.
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        if (kk + 1 < KK)
            read(stage, kk + 1, fa[(kk + 1) & 1]);
        mfmas(fa[kk & 1], kk);
        if (kk + 1 < KK)
            __builtin_amdgcn_sched_group_barrier(0x100, C::FM, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, C::FM * C::FN, 0);
    }
}

template <class C, bool ALIGNED, int KIND>
__global__ void __launch_bounds__(C::NT, C::OCC) k_gemm_packed(LayerDesc d)
{
    __shared__ v4i sm[C::SM];
    int tm, tn;
    tile_coords(xcd_remap(blockIdx.x, gridDim.x), d.tiles_m, d.tiles_n, tm, tn);
    const int m0 = tm * C::BM, n0 = tn * C::BN;
    v16i acc[C::FM][C::FN];
    mainloop_packed<C, ALIGNED, KIND>(d, keep_mask_dword(d.bits), m0, n0, acc, sm);
    epilogue<C>(d, m0, n0, acc, d.bits, reinterpret_cast<char *>(sm));
}

// Grouped step over every layer (see k_masked_gemm_grouped); every layer
// carries its packed weights.
template <class C, bool CONV>
__global__ void __launch_bounds__(C::NT, C::OCC)
k_gemm_packed_grouped(const LayerDesc *__restrict__ descs, int L, const uint8_t *table, int S,
                      int stage)
{
    __shared__ v4i sm[C::SM];
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
    const int bits = table[d.layer * S + stage];
    const uint32_t wmask = keep_mask_dword(bits);
    int tm, tn;
    tile_coords(t - d.tile_begin + d.tile_first, d.tiles_m, d.tiles_n, tm, tn);
    const int m0 = tm * C::BM, n0 = tn * C::BN;
    v16i acc[C::FM][C::FN];
    if (CONV && d.kind == KIND_CONV3X3)
        mainloop_packed<C, true, KIND_CONV3X3>(d, wmask, m0, n0, acc, sm);
    else
        mainloop_packed<C, true, KIND_LINEAR>(d, wmask, m0, n0, acc, sm);
    epilogue<C>(d, m0, n0, acc, bits, reinterpret_cast<char *>(sm));
}

template <class C>
hipError_t launch_packed_single(const LayerDesc &din, bool aligned, hipStream_t stream)
{
    LayerDesc d = din;
    fill_tiles<C>(d);
    const long long grid = (long long)d.tiles_m * d.tiles_n;
    if (grid > 0x7fffffffLL)
        return hipErrorInvalidValue;
    dim3 g((unsigned)grid), b(C::NT);
    if (d.kind == KIND_CONV3X3) {
        if (aligned)
            hipLaunchKernelGGL((k_gemm_packed<C, true, KIND_CONV3X3>), g, b, 0, stream, d);
        else
            hipLaunchKernelGGL((k_gemm_packed<C, false, KIND_CONV3X3>), g, b, 0, stream, d);
    } else if (aligned) {
        hipLaunchKernelGGL((k_gemm_packed<C, true, KIND_LINEAR>), g, b, 0, stream, d);
    } else {
        hipLaunchKernelGGL((k_gemm_packed<C, false, KIND_LINEAR>), g, b, 0, stream, d);
    }
    return hipGetLastError();
}

template <class C>
hipError_t launch_packed_grouped(const LayerDesc *d_descs, int L, int total_tiles,
                                 const uint8_t *d_table, int S, int stage, bool any_conv,
                                 hipStream_t stream)
{
    dim3 g((unsigned)total_tiles), b(C::NT);
    if (any_conv)
        hipLaunchKernelGGL((k_gemm_packed_grouped<C, true>), g, b, 0, stream, d_descs, L,
                           d_table, S, stage);
    else
        hipLaunchKernelGGL((k_gemm_packed_grouped<C, false>), g, b, 0, stream, d_descs, L,
                           d_table, S, stage);
    return hipGetLastError();
}

// Dispatch entry of one packed-weight tile configuration.
#define TASQ_DEFINE_PACKED_TILE(NAME, CFG)                                                    \
    const PackedTileOps &NAME()                                                               \
    {                                                                                         \
        static const PackedTileOps ops = {{CFG::BM, CFG::BN, CFG::BK},                        \
                                          &launch_packed_single<CFG>,                         \
                                          &launch_packed_grouped<CFG>, nullptr};              \
        return ops;                                                                           \
    }

}  // namespace tasq
