// Persistent grouped step with deep operand prefetch (256x256 tiles, 8 waves).
//
// Same operation and epilogue as k_masked_gemm_persistent (gemm_core.h):
// acc = X * W_b^T with W_b = W & keep_mask(b) (TASQ Sec. 3.2.1 Eq.
// lsb_masking, App. G.2 Eq. hw_rightshift), one grouped launch per denoising
// step, b from the (layer, stage) table.  What differs is how operands reach
// LDS, so that global loads have two K tiles of matrix work to land instead
// of one:
//   * activation tiles go from global memory straight to LDS
//     (buffer_load_dwordx4 ... lds: lane l of an instruction writes its 16
//     bytes at M0 + 16 l), three LDS stages, issued two K tiles ahead; the
//     XOR swizzle of the LDS rows is realised by the choice of global chunk
//     each lane fetches;
//   * weight tiles pass through registers, where the LSB mask is applied,
//     two K tiles in flight (a ring of two register slots), two LDS stages;
//   * LDS: 3 x 32 KiB of activations + 2 x 32 KiB of weights = 160 KiB.
// K tiles are numbered continuously across the tiles a workgroup walks, so
// the stage a K tile uses (g % 3, g % 2) rotates across tile boundaries and
// the next tile's first two K tiles are requested before the current tile's
// output stores: on gfx9 one in-order counter covers loads and stores, and
// loads issued behind 128 stores would wait for all of them.
//
// Barriers are plain s_barrier with the waits spelled out: a workgroup fence
// would wait for every direct-to-LDS load in flight (vmcnt(0)), which is the
// latency this schedule exists to hide.
#pragma once

#include <type_traits>

#include "gemm_core.h"

namespace tasq {

typedef __attribute__((address_space(3))) void lds_void_t;

namespace pers {

constexpr int kAStages = 3, kBStages = 2;

// s_waitcnt vmcnt(N) lgkmcnt(0) (gfx9 encoding: vmcnt[3:0] in bits 3:0,
// vmcnt[5:4] in bits 15:14, expcnt bits 6:4 left at 7, lgkmcnt bits 11:8 = 0).
template <int N>
__device__ __forceinline__ void wait_vm_lgkm0()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4));
}

// s_waitcnt lgkmcnt(0) alone (vmcnt and expcnt fields at their maxima): this
// wave's LDS reads and writes are done, its global requests may still be in
// flight.
__device__ __forceinline__ void wait_lgkm0()
{
    __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4));
}

// Workgroup barrier with no implied waits (the caller has issued them); the
// memory clobber keeps LDS accesses on their side of it.
__device__ __forceinline__ void barrier()
{
    asm volatile("s_barrier" ::: "memory");
}

}  // namespace pers

template <class C>
struct PersOperands {
    static_assert(C::BM == 256 && C::BN == 256 && C::BK == 128 && C::NT == 512,
                  "the direct-staged persistent step is written for 256x256x128, 8 waves");
    static constexpr int A_STAGE = C::BM * C::BK;       // bytes
    static constexpr int B_STAGE = C::BN * C::BK;
    static constexpr int LDS = pers::kAStages * A_STAGE + pers::kBStages * B_STAGE;
    static constexpr int A_LOADS = C::A_LOADS;          // direct loads per thread per K tile
    static constexpr int B_LOADS = C::B_LOADS;          // 16-byte weight chunks per thread
    static constexpr int KK = C::BK / 32;
    static constexpr int WRITE_KK = KK - 2;

    rsrc_t rX, rW;
    uint32_t offA, offB;      // global byte offsets of this thread's first chunks at k = 0
    uint32_t rowstep;         // 64 rows of K bytes: between a thread's successive chunks
    int K, nk;

    // Direct chunk i of wave w fills LDS chunks q = (8 i + w) * 64 + lane of
    // a stage: row q / 8 = 64 i + 8 w + lane / 8, physical 16-byte column
    // lane % 8, holding the logical column swz(row, lane % 8) (the swizzle
    // is an involution, and depends on the row only through row % 16, which
    // is the same for every i).  Weight chunk i of thread tid is row
    // tid / 8 + 64 i, column tid % 8.  Rows past M (N) fall at or past the
    // end of the buffer and read zero.
    __device__ __forceinline__ void init(const LayerDesc &d, int m0, int n0, int tid)
    {
        K = d.K;
        nk = (d.K + C::BK - 1) / C::BK;
        rX = make_rsrc(d.X, (uint32_t)d.M * (uint32_t)d.K);
        rW = make_rsrc(d.W, (uint32_t)d.N * (uint32_t)d.K);
        rowstep = 64u * (uint32_t)d.K;
        const int lane = tid & 63, wave = tid >> 6;
        const int ra = 8 * wave + lane / 8;
        offA = (uint32_t)(m0 + ra) * (uint32_t)d.K + (uint32_t)(16 * swz<C::CPR>(ra, lane % 8));
        offB = (uint32_t)(n0 + tid / 8) * (uint32_t)d.K + (uint32_t)(16 * (tid % 8));
    }

    // Activation K tile t (bytes t*BK ..) into LDS stage `base`.  Chunks past
    // K within a row read the next row's bytes, which meet zero weights; a K
    // tile past the layer's last (requested so that every wait sees the same
    // count) reads zero without touching memory.
    __device__ __forceinline__ void issue_a(char *base, int t) const
    {
        const int wave = threadIdx.x >> 6;
        // An opaque copy: the four offsets are formed here with one add each
        // rather than kept live through the main loop.
        uint32_t o = t < nk ? offA + (uint32_t)t * C::BK : kOOB;
        asm volatile("" : "+v"(o));
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rX, (lds_void_t *)(base + (8 * i + wave) * 1024), 16, o + (uint32_t)i * rowstep,
                0, 0, 0);
    }

    // Weight K tile t into a register slot; chunks at or past K read zero.
    __device__ __forceinline__ void load_b(v4i (&slot)[B_LOADS], int t) const
    {
        const uint32_t kt = (uint32_t)t * C::BK;
        const bool in_k = (int)kt + 16 * (int)(threadIdx.x % C::CPR) < K;
        uint32_t o = offB + kt;
        asm volatile("" : "+v"(o));
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i)
            slot[i] = ld16(rW, in_k ? o + (uint32_t)i * rowstep : kOOB);
    }

    // Masked weight slot into LDS stage sB (row-major rows of BK bytes,
    // swizzled like the activation rows).
    __device__ __forceinline__ static void store_b(const v4i (&slot)[B_LOADS], v4i *sB,
                                                   uint32_t wmask)
    {
        const int msk = (int)wmask;
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) {
            const int id = threadIdx.x + i * C::NT;
            const int r = id / C::CPR, c = id % C::CPR;
            v4i v = slot[i];
            v.x &= msk;
            v.y &= msk;
            v.z &= msk;
            v.w &= msk;
            sB[r * C::CPR + swz<C::CPR>(r, c)] = v;
        }
    }
};

// The epilogue's per-column factors (as epilogue_cols in gemm_core.h), in
// two parts: the loads, issued early and read with buffer loads (a
// generic-pointer load would also count as an LDS access and be waited for
// with every other memory request in flight), and the arithmetic, done when
// the epilogue needs it, so that the loads' latency is not waited for at
// the point of issue.
template <class C>
struct ColLoads {
    float sw[C::FN], bias[C::FN], wz[C::FN];
    int cs[C::FN];
    float alpha, zx;
};

template <class C, bool EXTRAS = false>
__device__ __forceinline__ void cols_request(const LayerDesc &d, int n0, int bits,
                                             ColLoads<C> &cl)
{
    const int lane = threadIdx.x & 63;
    const int wn = (threadIdx.x >> 6) % C::WAVES_N;
    const uint32_t nb = (uint32_t)d.N * 4u;
    const rsrc_t rsw = make_rsrc(d.sw, d.sw ? nb : 0u);
    const rsrc_t rbias = make_rsrc(d.bias, d.bias ? nb : 0u);
    const rsrc_t rcs = make_rsrc(d.colsums, d.act ? 8u * nb : 0u);
    const rsrc_t ract = make_rsrc(d.act, d.act ? 8u : 0u);
    cl.alpha = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(ract, 0, 0, 0));
    cl.zx = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(ract, 4, 0, 0));
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
        const int n = n0 + wn * C::WTN + j * 32 + (lane & 31);
        const bool nok = n < d.N;
        const uint32_t on = nok ? (uint32_t)n * 4u : kOOB;
        cl.sw[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsw, on, 0, 0));
        cl.bias[j] =
            __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rbias, on, 0, 0));
        cl.cs[j] = (int)__builtin_amdgcn_raw_buffer_load_b32(
            rcs, nok ? ((uint32_t)(bits - 1) * (uint32_t)d.N + (uint32_t)n) * 4u : kOOB, 0, 0);
        cl.wz[j] = 0.f;
        if constexpr (EXTRAS) {
            // weight zero points z_n, read only when the epilogue adds their term
            const rsrc_t rwz = make_rsrc(d.wz, d.wz && d.y ? nb : 0u);
            cl.wz[j] =
                __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rwz, on, 0, 0));
        }
    }
}

template <class C, bool EXTRAS = false>
__device__ __forceinline__ void cols_finish(const LayerDesc &d, int m0, int n0,
                                            const ColLoads<C> &cl, EpiCols<C> &ec)
{
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
    const int mrow = m0 + wm * C::WTM + 4 * (lane >> 5);
    const bool asym = d.act != nullptr;
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
        const int n = n0 + wn * C::WTN + j * 32 + (lane & 31);
        const bool nok = n < d.N;
        ec.scale[j] = (asym ? cl.alpha : d.sx) * cl.sw[j];
        ec.bias[j] = cl.bias[j];
        ec.corr[j] = asym ? (128.0f - cl.zx) * (float)cl.cs[j] : 0.0f;
        // (128 - z_n) times the column scale: the weight zero point's term
        ec.wsc[j] = EXTRAS && d.wz && d.y ? (128.0f - cl.wz[j]) * ec.scale[j] : 0.f;
        ec.base[j] = nok ? ((uint32_t)mrow * (uint32_t)d.N + (uint32_t)n) * 4u : kOOB;
    }
}

// One workgroup per compute unit walks its XCD's run of work units (as in
// k_masked_gemm_persistent).  g counts K tiles across the walk: K tile t of
// the current tile is global K tile g0 + t, in activation stage (g0+t) % 3
// and weight stage (g0+t) % 2; weight K tile t sits in register slot t % 2
// from its load until its LDS store (both slots are empty at a tile
// boundary, so the slots need not rotate across tiles).
template <class C, bool EXTRAS>
__global__ void __launch_bounds__(C::NT, C::OCC)
k_masked_gemm_persistent_ds(const LayerDesc *__restrict__ descs, int L, int total, XcdRuns runs,
                            const uint8_t *__restrict__ table, int S, int stage, int parties)
{
    using Ops = PersOperands<C>;
    __shared__ __attribute__((aligned(1024))) char sm[Ops::LDS];
    char *const smA = sm;
    char *const smB = sm + pers::kAStages * Ops::A_STAGE;
    constexpr int NX = 8;
    constexpr int KK = Ops::KK, WRITE_KK = Ops::WRITE_KK;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;

    const int wgs = gridDim.x / NX / parties;
    const int x = blockIdx.x % NX, j = blockIdx.x / NX;
    const int part = j % parties, jj = j / parties;
    const int xbeg = runs.begin[x], xend = runs.begin[x + 1];
    const int pspan = (xend - xbeg + parties - 1) / parties;
    const int ubeg = xbeg + part * pspan;
    const int uend = min(xend, ubeg + pspan);
    int u = ubeg + jj;
    if (u >= uend)
        return;

    auto bits_of = [&](int sg) {
        const int idx = descs[sg].layer * S + stage;
        const uint32_t w = reinterpret_cast<const uint32_t *>(table)[idx >> 2];
        return (int)((w >> (8 * (idx & 3))) & 0xffu);
    };
    auto a_stage = [&](int g) { return smA + (g % pers::kAStages) * Ops::A_STAGE; };
    auto b_stage = [&](int g) {
        return reinterpret_cast<v4i *>(smB + (g & 1) * Ops::B_STAGE);
    };

    Ops ops;
    v4i ring[2][Ops::B_LOADS];
    // A tile's first two K tiles: activations to LDS, weights to the ring.
    // Every request of the schedule is issued whether or not its K tile
    // exists (one past K reads zero weights, or activation bytes of other
    // rows into a stage no K tile of this tile reads), so that the count of
    // requests in flight is the same at every wait.
    auto issue_first = [&](int g0, int t0) {
        ops.issue_a(a_stage(g0), t0);
        ops.load_b(ring[0], t0);
        ops.issue_a(a_stage(g0 + 1), t0 + 1);
        ops.load_b(ring[1], t0 + 1);
    };

    int seg = find_segment(descs, L, u);
    int m0, n0;
    unit_coords<C>(descs[seg], u, m0, n0);
    int bits = bits_of(seg);
    int g0 = 0;                       // global K tile of the current tile's K tile 0
    bool first = true;
    {
        const LayerDesc &d0 = descs[seg];
        ops.init(d0, m0, n0, tid);
        issue_first(0, 0);
    }
    for (;;) {
        const LayerDesc &d = descs[seg];
        const int nk = (d.K + C::BK - 1) / C::BK;
        const uint32_t wmask = keep_mask_dword(bits);

        // Prologue: weight K tile 0 to its stage (the wait for the slot also
        // covers the activation K tile 0 issued before it), weight K tile 2
        // requested into the freed slot.
        Ops::store_b(ring[0], b_stage(g0), wmask);
        ops.load_b(ring[0], 2);
        pers::wait_vm_lgkm0<63>();
        pers::barrier();

        v16i acc[C::FM][C::FN];
        zero_acc<C>(acc);
        v4i fa[2][C::FM], fb[2][C::FN];
        // Fragment reads: row wm*WTM + 32 i + lane%32 (activations) or
        // wn*WTN + 32 j + lane%32 (weights), logical 16-byte column
        // 2 kk + lane/32, physical column swz(row, that); the swizzle depends
        // on the row only through lane%16, so one lane offset per sub-step
        // serves every fragment and both operands.
        uint32_t lane_off[KK];
        {
            const int xr = (lane & 7) ^ ((lane >> 3) & 1);
#pragma unroll
            for (int kk = 0; kk < KK; ++kk)
                lane_off[kk] = (uint32_t)((lane & 31) * C::BK + 16 * ((2 * kk + (lane >> 5)) ^ xr));
        }
        auto read = [&](int g, int kk, v4i (&a)[C::FM], v4i (&b)[C::FN]) {
            const char *A = a_stage(g) + wm * C::WTM * C::BK + lane_off[kk];
            const char *B = reinterpret_cast<const char *>(b_stage(g)) + wn * C::WTN * C::BK +
                            lane_off[kk];
#pragma unroll
            for (int i = 0; i < C::FM; ++i)
                a[i] = *reinterpret_cast<const v4i *>(A + i * 32 * C::BK);
#pragma unroll
            for (int jx = 0; jx < C::FN; ++jx)
                b[jx] = *reinterpret_cast<const v4i *>(B + jx * 32 * C::BK);
        };
        auto mfmas = [&](v4i (&a)[C::FM], v4i (&b)[C::FN]) {
#pragma unroll
            for (int i = 0; i < C::FM; ++i)
#pragma unroll
                for (int jx = 0; jx < C::FN; ++jx)
                    acc[i][jx] =
                        __builtin_amdgcn_mfma_i32_32x32x32_i8(a[i], b[jx], acc[i][jx], 0, 0, 0);
        };

        // K tile t (not the last), its weight K tile t+1 in register slot V.
        auto ktile = [&](auto slot_tag, int t) {
            constexpr int slot = decltype(slot_tag)::value;
            const int g = g0 + t;
            // Activation K tile t+2 goes to the stage K tile t-1 used (every
            // wave finished reading it before the last barrier).
            ops.issue_a(a_stage(g + 2), t + 2);
#pragma unroll
            for (int kk = 0; kk + 1 < KK; ++kk) {
                read(g, kk + 1, fa[(kk + 1) & 1], fb[(kk + 1) & 1]);
                mfmas(fa[kk & 1], fb[kk & 1]);
                if (kk == WRITE_KK) {
                    // weight K tile t+1 to the other weight stage (read in
                    // K tile t-1, done before the last barrier), then the
                    // slot is refilled with K tile t+3.
                    Ops::store_b(ring[slot], b_stage(g + 1), wmask);
                    ops.load_b(ring[slot], t + 3);
                }
#pragma unroll
                for (int i = 0; i < C::FM * C::FN; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    if (i < C::FM + C::FN)
                        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                }
            }
            // Activation K tile t+1 landed (issued at the start of K tile
            // t-1, or with the tile's first loads): after it come weight K
            // tile t+2, activation K tile t+2 and weight K tile t+3, 12
            // requests.
            // Right after a tile boundary the previous tile's output stores
            // sit between them, well over the 63 requests a wave can have in
            // flight, so the hardware's own limit has already retired it.
            if (t == 0 && !first)
                pers::wait_vm_lgkm0<63>();
            else
                pers::wait_vm_lgkm0<12>();
            pers::barrier();
            read(g + 1, 0, fa[0], fb[0]);
            mfmas(fa[(KK - 1) & 1], fb[(KK - 1) & 1]);
#pragma unroll
            for (int i = 0; i < C::FM * C::FN; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                if (i < C::FM + C::FN)
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
        };

        read(g0, 0, fa[0], fb[0]);
        int t = 0;
        for (; t + 2 < nk; t += 2) {
            ktile(std::integral_constant<int, 1>{}, t);
            ktile(std::integral_constant<int, 0>{}, t + 1);
        }
        if (t + 1 < nk)
            ktile(std::integral_constant<int, 1>{}, t);
        // Before the last K tile's matrix work (its operands are already in
        // LDS): the epilogue's per-column factors are requested, and the
        // next tile's coordinates found and its first two K tiles requested,
        // so that all of these land under the last K tile's MFMAs.  The next
        // tile's stages are free: activation stages (g0+nk) % 3 and
        // (g0+nk+1) % 3 and weight stage (g0+nk) % 2 held K tiles nk-3 and
        // nk-2 (or the previous tile's), whose reads every wave finished
        // before the last barrier; the register slots hold only the requests
        // past K.
        ColLoads<C> cl;
        cols_request<C, EXTRAS>(d, n0, bits, cl);
        const LayerDesc &dc = d;
        const int mc = m0, nc = n0;
        const int g1 = g0 + nk;
        u += wgs;
        const bool more = u < uend;
        if (more) {
            seg = find_segment(descs, L, u);
            unit_coords<C>(descs[seg], u, m0, n0);
            bits = bits_of(seg);
            int t2 = tid;
            asm volatile("" : "+v"(t2));
            ops.init(descs[seg], m0, n0, t2);
        }
        // With no next tile the same requests go out past K (zeros into free
        // stages and slots), so that the epilogue's waits see one count.
        issue_first(g1, more ? 0 : nk);
        {
            const int g = g0 + nk - 1;
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                if (kk + 1 < KK)
                    read(g, kk + 1, fa[(kk + 1) & 1], fb[(kk + 1) & 1]);
                mfmas(fa[kk & 1], fb[kk & 1]);
                if (kk + 1 < KK)
                    __builtin_amdgcn_sched_group_barrier(0x100, C::FM + C::FN, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, C::FM * C::FN, 0);
            }
        }
        __builtin_amdgcn_sched_barrier(0);
        EpiCols<C> ec;
        cols_finish<C, EXTRAS>(dc, mc, nc, cl, ec);
        // The low-rank and weight-zero-point operands of the tile are staged
        // in the weight stages, idle from the last K tile's final LDS reads
        // (every wave's, after the first barrier) until the next tile's
        // prologue stores its weight K tile 0 (after the last barrier).
        bool staged = false;
        if constexpr (EXTRAS) {
            const bool lowrank = dc.lr_T != nullptr && dc.y != nullptr;
            const bool wzero = dc.wz != nullptr && dc.y != nullptr;
            staged = lowrank || wzero;
            if (staged) {
                pers::wait_lgkm0();
                pers::barrier();
                if (lowrank)
                    stage_lowrank<C>(dc, mc, nc, smB);
                if (wzero)
                    stage_rowsums<C>(dc, mc, smB);
                pers::wait_lgkm0();
                pers::barrier();
            }
        }
        epilogue_write<C, true, EXTRAS>(dc, acc, ec, smB);
        if (staged) {
            pers::wait_lgkm0();
            pers::barrier();
        }
        __builtin_amdgcn_sched_barrier(0);
        if (!more)
            break;
        g0 = g1;
        first = false;
    }
}

template <class C, bool EXTRAS>
hipError_t launch_persistent_ds_cfg(const LayerDesc *d_descs, int L, int total_tiles,
                                    const XcdRuns &runs, const uint8_t *d_table, int S, int stage,
                                    int wgs_per_xcd, int parties, hipStream_t stream)
{
    if (wgs_per_xcd < 1 || total_tiles < 1 || parties < 1 || wgs_per_xcd % parties != 0 ||
        !xcd_runs_valid(runs, total_tiles))
        return hipErrorInvalidValue;
    dim3 g((unsigned)(8 * wgs_per_xcd)), b(C::NT);
    hipLaunchKernelGGL((k_masked_gemm_persistent_ds<C, EXTRAS>), g, b, 0, stream, d_descs, L,
                       total_tiles, runs, d_table, S, stage, parties);
    return hipGetLastError();
}

#define TASQ_DEFINE_TILE_DS(NAME, CFG)                                                      \
    const TileOps &NAME()                                                                   \
    {                                                                                       \
        static const TileOps ops = {{CFG::BM, CFG::BN, CFG::BK}, &launch_single_cfg<CFG>,   \
                                    &launch_planes_cfg<CFG>, &launch_grouped_cfg<CFG>,      \
                                    &launch_split_cfg<CFG>,                                 \
                                    &launch_persistent_ds_cfg<CFG, false>,                  \
                                    &launch_persistent_ds_cfg<CFG, true>};                  \
        return ops;                                                                         \
    }

}  // namespace tasq
