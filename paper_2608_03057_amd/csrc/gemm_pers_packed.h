// Persistent grouped step on packed weights (256x256 tiles, 8 waves of
// 128x64): the weights come from the packed layout (gemm_packed.h) straight
// into registers, so LDS holds only activations, five stages of them.
//
// Same operation as k_masked_gemm_persistent_ds (gemm_pers.h): acc = X * W_b^T
// with W_b = W & keep_mask(b) (TASQ Sec. 3.2.1 Eq. lsb_masking, App. G.2 Eq.
// hw_rightshift), one launch per denoising step, b from the (layer, stage)
// table, one workgroup per compute unit walking its XCD's run of tiles.
// What differs is the operand flow:
//   * activation K tiles go straight to LDS (buffer_load_dwordx4 ... lds),
//     five 32 KiB stages, requested four K tiles ahead;
//   * each wave loads the packed weight fragments of its own 64 output
//     channels (one 16-byte load per lane and 32x32 fragment) one K tile
//     ahead into the registers the current K tile's matrix work has just
//     consumed, and masks them as it feeds them to the MFMAs;
//   * the request positions run ahead across tile boundaries: a walk over
//     the workgroup's units, K tile by K tile, for the activations (four
//     ahead) and one for the weights (one ahead), so the next tile's first
//     operands are in flight while the current tile finishes.
// Every K tile issues the same requests in the same order (walks past the
// last unit request zero-reads into a stage nothing reads again), so the
// wait before each barrier is a fixed count, or the hardware's limit of 63
// right after a tile's 128 output stores per lane.
#pragma once

#include <type_traits>

#include "gemm_packed.h"
#include "gemm_pers.h"

namespace tasq {

namespace ppk {

constexpr int kAStages = 5;     // activation LDS stages
constexpr int kAhead = 4;       // activation K tiles requested ahead of the one computed
static_assert(kAStages == kAhead + 1, "one stage being read, the others in flight");

}  // namespace ppk

// A position in the workgroup's walk: unit u (segment seg, tile origin m0,
// n0) and K tile t of its nk; live while u is below the run's end.
struct KPos {
    int u, seg, m0, n0, t, nk;
    bool live;
};

template <class C>
__device__ __forceinline__ void kpos_enter(const LayerDesc *__restrict__ descs, int L, int uend,
                                           KPos &p)
{
    p.t = 0;
    p.live = p.u < uend;
    if (!p.live) {
        p.nk = 1;
        return;
    }
    p.seg = find_segment(descs, L, p.u);
    unit_coords<C>(descs[p.seg], p.u, p.m0, p.n0);
    // (a layer with K = 0 still takes one K tile, of zero operands, so that
    // its outputs are written)
    p.nk = max(1, (descs[p.seg].K + C::BK - 1) / C::BK);
}

// Advances by one K tile; returns whether the position entered a new unit.
template <class C>
__device__ __forceinline__ bool kpos_next(const LayerDesc *__restrict__ descs, int L, int uend,
                                          int step, KPos &p)
{
    if (!p.live)
        return false;
    if (++p.t < p.nk)
        return false;
    p.u += step;
    kpos_enter<C>(descs, L, uend, p);
    return true;
}

template <class C>
__global__ void __launch_bounds__(C::NT, C::OCC)
k_gemm_packed_persistent(const LayerDesc *__restrict__ descs, int L, int total, XcdRuns runs,
                         const uint8_t *__restrict__ table, int S, int stage, int parties)
{
    static_assert(C::BM == 256 && C::BN == 256 && C::BK == 128 && C::NT == 512 && C::FN == 2,
                  "written for 256x256x128 tiles of 8 waves (128x64 per wave)");
    using AOps = PersOperands<C>;
    constexpr int A_STAGE = C::BM * C::BK;
    __shared__ __attribute__((aligned(1024))) char sm[ppk::kAStages * A_STAGE];
    constexpr int NX = 8;
    constexpr int KK = C::KK;
    constexpr int RA = C::A_LOADS, RB = C::FN;    // requests per K tile: activation, per sub-step
    // Requests after activation K tile g+1 at the barrier of K tile g: the
    // rest of the prologue's activation requests (for g < kAhead-2), the
    // whole K tiles since (RB KK weight and RA activation requests each; at
    // most kAhead-2) and this K tile's first RB (KK-1) weight requests.
    constexpr auto wait_count = [](int g) constexpr {
        constexpr int KKc = C::KK;
        const int rest = g < ppk::kAhead - 2 ? ppk::kAhead - 2 - g : 0;
        const int whole = g < ppk::kAhead - 2 ? g : ppk::kAhead - 2;
        return rest * RA + whole * (RA + RB * KKc) + RB * (KKc - 1);
    };
    static_assert(ppk::kAhead == 4, "the waits below spell out g = 0, 1 and the steady state");
    static_assert(wait_count(2) < 64, "fits the counter");
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
    if (ubeg + jj >= uend)
        return;

    auto bits_of = [&](int sg) {
        const int idx = descs[sg].layer * S + stage;
        const uint32_t w = reinterpret_cast<const uint32_t *>(table)[idx >> 2];
        return (int)((w >> (8 * (idx & 3))) & 0xffu);
    };
    auto a_stage = [&](int g) { return sm + (g % ppk::kAStages) * A_STAGE; };

    // Compute position, weight request position (one K tile ahead) and
    // activation request position (kAhead ahead).
    KPos pc, pb, pa;
    pc.u = pb.u = pa.u = ubeg + jj;
    kpos_enter<C>(descs, L, uend, pc);
    pb = pc;
    pa = pc;

    // Activation requests of the position pa (zero-reads once it is past
    // the run), then one step.
    AOps aops;
    auto a_reload = [&]() {
        if (pa.live)
            aops.init(descs[pa.seg], pa.m0, pa.n0, tid);
        else
            aops.nk = 0;
    };
    a_reload();
    int ga = 0;                      // global K tile of position pa
    auto a_issue = [&]() {
        aops.issue_a(a_stage(ga), pa.live ? pa.t : 1);
        ++ga;
        if (kpos_next<C>(descs, L, uend, wgs, pa))
            a_reload();
    };

    // Weight fragments of position pb, sub-step kk, into wb[.][kk].
    rsrc_t rW;
    uint32_t offB[C::FN];
    auto b_reload = [&]() {
        if (pb.live) {
            const LayerDesc &d = descs[pb.seg];
            const int KS = (d.K + 127) / 128 * 4;
            const int NB = (d.N + 31) / 32;
            rW = make_rsrc(d.Wp, (uint32_t)packed_weight_bytes(d.N, d.K));
#pragma unroll
            for (int jx = 0; jx < C::FN; ++jx) {
                const int nb = (pb.n0 + wn * C::WTN) / 32 + jx;
                offB[jx] = nb < NB ? (uint32_t)nb * (uint32_t)KS * 1024u + (uint32_t)lane * 16u
                                   : kOOB;
            }
        } else {
            rW = make_rsrc(nullptr, 0u);
#pragma unroll
            for (int jx = 0; jx < C::FN; ++jx)
                offB[jx] = kOOB;
        }
    };
    b_reload();
    v4i wb[C::FN][KK];
    auto b_load = [&](int kk) {
        const uint32_t step = (uint32_t)(pb.live ? pb.t * KK + kk : 0) * 1024u;
#pragma unroll
        for (int jx = 0; jx < C::FN; ++jx) {
            uint32_t o = offB[jx] == kOOB ? kOOB : offB[jx] + step;
            asm volatile("" : "+v"(o));
            wb[jx][kk] = ld16(rW, o);
        }
    };
    auto b_next = [&]() {
        if (kpos_next<C>(descs, L, uend, wgs, pb))
            b_reload();
    };

    // Prologue: weight K tile 0, then activation K tiles 0 .. kAhead-1 of
    // the walk (the order a K tile ends with, so that the compiler's waits
    // for weight fragments in the loop see the steady-state counts).
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
        b_load(kk);
    b_next();
#pragma unroll
    for (int i = 0; i < ppk::kAhead; ++i)
        a_issue();

    // Fragment reads: as in k_masked_gemm_persistent_ds.
    uint32_t lane_off[KK];
    {
        const int xr = (lane & 7) ^ ((lane >> 3) & 1);
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
            lane_off[kk] = (uint32_t)((lane & 31) * C::BK + 16 * ((2 * kk + (lane >> 5)) ^ xr));
    }
    v4i fa[2][C::FM];
    auto read = [&](int g, int kk, v4i (&a)[C::FM]) {
        const char *A = a_stage(g) + wm * C::WTM * C::BK + lane_off[kk];
#pragma unroll
        for (int i = 0; i < C::FM; ++i)
            a[i] = *reinterpret_cast<const v4i *>(A + i * 32 * C::BK);
    };
    v16i acc[C::FM][C::FN];
    uint32_t wmask = keep_mask_dword(bits_of(pc.seg));
    auto mfmas = [&](v4i (&a)[C::FM], int kk) {
        const int msk = (int)wmask;
#pragma unroll
        for (int jx = 0; jx < C::FN; ++jx) {
            v4i w = wb[jx][kk];
            w.x &= msk;
            w.y &= msk;
            w.z &= msk;
            w.w &= msk;
#pragma unroll
            for (int i = 0; i < C::FM; ++i)
                acc[i][jx] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[i], w, acc[i][jx], 0, 0, 0);
        }
    };
    auto group_order = [&]() {
#pragma unroll
        for (int i = 0; i < C::FM * C::FN; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            if (i < C::FM)
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
    };

    zero_acc<C>(acc);
    int g = 0;                       // global K tile of position pc
    int epi_age = ppk::kAhead - 1;   // K tiles since the last tile's stores, less one (capped)
    // Activation K tile 0 landed: after it come K tiles 1 .. kAhead-1.
    pers::wait_vm_lgkm0<(ppk::kAhead - 1) * RA>();
    pers::barrier();
    read(0, 0, fa[0]);
    ColLoads<C> cl;
    for (;;) {
        const bool last = pc.t + 1 == pc.nk;
        // (a tile of one K tile: its column factors now; otherwise at the
        // end of its second-to-last K tile, below)
        if (last && pc.nk == 1)
            cols_request<C>(descs[pc.seg], pc.n0, bits_of(pc.seg), cl);
#pragma unroll
        for (int kk = 0; kk + 1 < KK; ++kk) {
            read(g, kk + 1, fa[(kk + 1) & 1]);
            mfmas(fa[kk & 1], kk);
            b_load(kk);
            group_order();
        }
        // Activation K tile g+1 landed.  It was requested at the end of K
        // tile g+1-kAhead (or in the prologue); the requests after it are
        // wait_count(g).  Within kAhead-1 K tiles of a tile's output stores
        // the count is past the 63 a wave can have in flight.
        if (epi_age < ppk::kAhead - 1)
            pers::wait_vm_lgkm0<63>();
        else if (g == 0)
            pers::wait_vm_lgkm0<wait_count(0)>();
        else if (g == 1)
            pers::wait_vm_lgkm0<wait_count(1)>();
        else
            pers::wait_vm_lgkm0<wait_count(2)>();
        pers::barrier();
        read(g + 1, 0, fa[0]);
        mfmas(fa[(KK - 1) & 1], KK - 1);
        b_load(KK - 1);
        b_next();
        // The activation request goes after this K tile's weight requests:
        // the counter is in order, so a wait for a weight fragment would
        // otherwise wait for the activation K tiles requested before it.
        if (pc.t + 2 == pc.nk)
            cols_request<C>(descs[pc.seg], pc.n0, bits_of(pc.seg), cl);
        a_issue();
        group_order();
        epi_age = epi_age < ppk::kAhead - 1 ? epi_age + 1 : ppk::kAhead - 1;
        if (last) {
            __builtin_amdgcn_sched_barrier(0);
            const LayerDesc &dc = descs[pc.seg];
            EpiCols<C> ec;
            cols_finish<C>(dc, pc.m0, pc.n0, cl, ec);
            epilogue_write<C, true, false>(dc, acc, ec, reinterpret_cast<const char *>(sm));
            __builtin_amdgcn_sched_barrier(0);
            epi_age = 0;
            zero_acc<C>(acc);
        }
        ++g;
        kpos_next<C>(descs, L, uend, wgs, pc);
        if (!pc.live)
            break;
        if (pc.t == 0)
            wmask = keep_mask_dword(bits_of(pc.seg));
    }
}

template <class C>
hipError_t launch_packed_persistent(const LayerDesc *d_descs, int L, int total_tiles,
                                    const XcdRuns &runs, const uint8_t *d_table, int S, int stage,
                                    int wgs_per_xcd, int parties, hipStream_t stream)
{
    if (wgs_per_xcd < 1 || total_tiles < 1 || parties < 1 || wgs_per_xcd % parties != 0 ||
        !xcd_runs_valid(runs, total_tiles))
        return hipErrorInvalidValue;
    dim3 g((unsigned)(8 * wgs_per_xcd)), b(C::NT);
    hipLaunchKernelGGL((k_gemm_packed_persistent<C>), g, b, 0, stream, d_descs, L, total_tiles,
                       runs, d_table, S, stage, parties);
    return hipGetLastError();
}

// Dispatch entry of the 256x256 packed-weight tile with its persistent step.
#define TASQ_DEFINE_PACKED_TILE_PERS(NAME, CFG)                                               \
    const PackedTileOps &NAME()                                                               \
    {                                                                                         \
        static const PackedTileOps ops = {{CFG::BM, CFG::BN, CFG::BK},                        \
                                          &launch_packed_single<CFG>,                         \
                                          &launch_packed_grouped<CFG>,                        \
                                          &launch_packed_persistent<CFG>};                    \
        return ops;                                                                           \
    }

}  // namespace tasq
