// Masked int8 GEMM for gfx950 (CDNA4).
//
// acc[m][n] = sum_k X[m][k] * W_b[n][k],  W_b = W & keep_mask(b)
// y[m][n]   = float(acc) * (sx * sw[n]) (+ bias[n])
//
// The LSB mask (TASQ Sec. 3.2.1 Eq. lsb_masking, App. G.2 Eq. hw_rightshift)
// is one v_and_b32 per four weights, applied while a weight tile passes
// through registers between the global load and the LDS store; the MFMA
// main loop never sees an unmasked weight and never depends on b, so one
// compiled kernel serves every precision (App. G.1).
//
// Structure:
//   * block tile BM x BN over (M, N), K consumed in BK-byte steps;
//   * global -> VGPR (16-byte loads, mask on the weight side) -> LDS, two
//     LDS stages and a ring of PF K tiles in flight in registers, one barrier
//     per K step placed so that MFMAs cover it (see mainloop);
//   * LDS rows of BK bytes, 16-byte chunks XOR-swizzled so that the 32 rows
//     one MFMA operand read touches fall in distinct banks;
//   * each wave owns a (BM/WAVES_M) x (BN/WAVES_N) sub-tile of
//     v_mfma_i32_32x32x32_i8 accumulators (int32, exact);
//   * epilogue straight from the accumulators: lane l of a 32x32 block holds
//     column l%32, so every store instruction writes full 128-byte row
//     segments.
#pragma once

#include "tasq_internal.h"

namespace tasq {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

// LDS row pitch of the low-rank branch's staged operands: a rank-32 row of
// bfloat16 plus 16 bytes, so that the 16-byte fragment reads of 8
// consecutive rows fall in distinct banks.
constexpr int kLrPitch = 2 * kLowrankMaxRank + 16;

template <int BM_, int BN_, int BK_, int WAVES_M_, int WAVES_N_, int PF_ = 2, int OCC_ = 2>
struct Cfg {
    static constexpr int OCC = OCC_;                    // target waves per SIMD
    static constexpr int NSTAGE = 2;                    // K tiles resident in LDS
    static constexpr int BM = BM_, BN = BN_, BK = BK_;
    static constexpr int WAVES_M = WAVES_M_, WAVES_N = WAVES_N_;
    static constexpr int PF = PF_;                      // K tiles in flight in registers
    static constexpr int NT = WAVES_M * WAVES_N * 64;
    static constexpr int WTM = BM / WAVES_M, WTN = BN / WAVES_N;
    static constexpr int FM = WTM / 32, FN = WTN / 32;
    static constexpr int CPR = BK / 16;                 // 16-byte chunks per row
    static constexpr int A_LOADS = BM * CPR / NT;
    static constexpr int B_LOADS = BN * CPR / NT;
    // LDS of the A operand, also holding the epilogue's staged operands:
    // T rows as bfloat16 hi and lo parts, rows of U, then one fp32 row term
    // per tile row (the weight zero point's activation sums).
    static constexpr int LR_BYTES = (2 * BM + BN) * kLrPitch + 4 * BM;
    static constexpr int SMA = NSTAGE * BM * CPR > (LR_BYTES + 15) / 16 ? NSTAGE * BM * CPR
                                                                       : (LR_BYTES + 15) / 16;
    static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile must hold 32x32 blocks");
    static_assert(BK % 32 == 0 && (CPR == 4 || CPR == 8), "BK must be 64 or 128");
    static_assert((BM * CPR) % NT == 0 && (BN * CPR) % NT == 0, "loads must divide");
    static_assert(BK / 32 % 2 == 0, "an even number of 32-wide sub-steps per K tile");
};

// Physical 16-byte chunk of logical chunk c in LDS row r.  For 128-byte rows
// (8 chunks) rows 0..7 map a fixed c to 8 distinct chunks, and rows of equal
// parity among 0..15 as well, so a 32-row operand read is conflict free for
// both 128-byte and 256-byte bank windows; likewise for 64-byte rows.
template <int CPR>
__device__ __forceinline__ int swz(int r, int c)
{
    if constexpr (CPR == 8)
        return c ^ ((r & 7) ^ ((r >> 3) & 1));
    else
        return c ^ (((r >> 1) ^ (r >> 3)) & 3);
}

// ---------------------------------------------------------------- buffers

// Raw buffer resources: a load whose byte offset is at or past num_records
// returns zero and such a store is dropped, which bounds every access to
// its operand without per-element checks.  Offsets are 32-bit; the host
// keeps every operand below 2 GiB and kOOB marks a lane with nothing to do.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t kOOB = 0x80000000u;

__device__ __forceinline__ rsrc_t make_rsrc(const void *p, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes,
                                             0x00020000);
}

__device__ __forceinline__ v4i ld16(rsrc_t r, uint32_t off)
{
    return __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

__device__ __forceinline__ v2i ld8(rsrc_t r, uint32_t off)
{
    return __builtin_bit_cast(v2i, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}

// Output stores carry the non-temporal hint (cache-policy bit 1 on gfx950):
// the outputs are written once and never re-read by the kernel, and without
// the hint they evict the activation and weight tiles that neighbouring
// workgroups are still reading from L2.
__device__ __forceinline__ void st32(rsrc_t r, uint32_t off, uint32_t v)
{
    __builtin_amdgcn_raw_buffer_store_b32(v, r, off, 0, 2);
}

// A cacheable store, for data re-read right after (split-K partials).
__device__ __forceinline__ void st32_cached(rsrc_t r, uint32_t off, uint32_t v)
{
    __builtin_amdgcn_raw_buffer_store_b32(v, r, off, 0, 0);
}

__device__ __forceinline__ v4i zero4() { return v4i{0, 0, 0, 0}; }

// ------------------------------------------------- fallback (unaligned) loads

// 16 bytes at p[0..15]; bytes with index >= valid read as zero.
__device__ __forceinline__ v4i load_bytes(const int8_t *p, int valid)
{
    uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < 16; ++i)
        if (i < valid)
            w[i >> 2] |= (uint32_t)(uint8_t)p[i] << (8 * (i & 3));
    return v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
}

// Chunk (row, kbyte..kbyte+15) of a row-major [rows][K] int8 matrix, any K.
__device__ __forceinline__ v4i load_rowmajor_any(const int8_t *base, int rows, int K, int row,
                                                 int kbyte)
{
    if (row >= rows || kbyte >= K)
        return zero4();
    return load_bytes(base + (size_t)row * (size_t)K + kbyte, K - kbyte);
}

// Chunk of the implicit-GEMM activation of a 3x3 / pad 1 conv for any C:
// element k of row m = h*Wd + w is X[h + r - 1][w + s - 1][ci] with
// k = (r*3 + s)*C + ci, or 0 in the padding.
__device__ __forceinline__ v4i load_conv_any(const LayerDesc &d, int m, int kbyte)
{
    if (m >= d.M || kbyte >= d.K)
        return zero4();
    uint32_t w[4] = {0, 0, 0, 0};
    const int h = m / d.Wd, x = m - (m / d.Wd) * d.Wd;
    for (int i = 0; i < 16 && kbyte + i < d.K; ++i) {
        const int k = kbyte + i;
        const int tap = k / d.C, ci = k - (k / d.C) * d.C;
        const int hh = h + tap / 3 - 1, ww = x + tap % 3 - 1;
        if (hh >= 0 && hh < d.H && ww >= 0 && ww < d.Wd)
            w[i >> 2] |= (uint32_t)(uint8_t)d.X[((size_t)hh * d.Wd + ww) * (size_t)d.C + ci]
                         << (8 * (i & 3));
    }
    return v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
}

// ----------------------------------------------------------- bit planes

// Plane words are stored rotated (tasq_pack_planes): element (group g, byte
// c) of plane p's word sits at bit (8c + g + p) mod 32, so for one group the
// planes' bits land on disjoint positions 0x01010101 << ((g + p) % 8).
// plane_bits adds plane p's bits of group g to a merged word with one
// v_and_or_b32; plane_place rotates the merged word right by g, which puts
// bit p of each of the group's four codes at bit p of bytes 0..3.
__device__ __forceinline__ uint32_t plane_bits(uint32_t word, int g, int p, uint32_t merged)
{
    uint32_t r = (word & (0x01010101u << ((g + p) & 7))) | merged;
    // An empty register barrier: left to itself the compiler re-associates
    // a chain of these into separate ANDs and three-input ORs (about 1.5
    // instructions per plane instead of one v_and_or_b32).  The instruction
    // itself stays compiler-generated, so the wait states that a VALU result
    // needs before a matrix instruction reads it are still inserted.
    asm("" : "+v"(r));
    return r;
}

__device__ __forceinline__ uint32_t plane_place(uint32_t merged, int g)
{
    return __builtin_amdgcn_alignbit(merged, merged, (uint32_t)g);
}

// Bytes of the bit-plane buffer of an [N][K] weight (tasq_pack_planes): 8
// planes x 32 * ceil(N/32) channels x ceil(K/128) blocks x 16 bytes.
__host__ __device__ inline size_t planes_bytes(int N, int K)
{
    return (size_t)8 * (size_t)((N + 31) / 32) * 32 * (size_t)((K + 127) / 128) * 16;
}

// Chunk (row n, kbyte..kbyte+15, kbyte a multiple of 16) of W_b rebuilt from
// the top b bit planes (App. G.2: the b-bit operand is the top b planes of
// the stored buffer; the dropped planes are never read).  Plane q holds bit
// 7 - q of each code; the result is the two's-complement byte of W_b.  Word
// w of channel n = 32 nb + 16 f + r in block kb of plane q is word
// ((nb * 8 + q) * KB + kb) * 128 + 8 r + 2 w + f.
__device__ __forceinline__ v4i load_planes(const uint32_t *P, int N, int K, int b, int n,
                                           int kbyte)
{
    if (n >= N || kbyte >= K)
        return zero4();
    const int KB = (K + 127) >> 7;
    const size_t plane_stride = (size_t)KB * 128;
    const int s = (kbyte & 127) >> 5, h = (kbyte >> 4) & 1;
    const uint32_t *base = P + ((size_t)(n >> 5) * 8 * KB + (size_t)(kbyte >> 7)) * 128 +
                           8 * (n & 15) + 2 * (2 * h + (s >> 1)) + ((n >> 4) & 1);
    const int g0 = 4 * (s & 1);
    uint32_t d0 = 0, d1 = 0, d2 = 0, d3 = 0;
    for (int q = 0; q < b; ++q) {
        const uint32_t w = base[q * plane_stride];
        const int p = 7 - q;
        d0 = plane_bits(w, g0 + 0, p, d0);
        d1 = plane_bits(w, g0 + 1, p, d1);
        d2 = plane_bits(w, g0 + 2, p, d2);
        d3 = plane_bits(w, g0 + 3, p, d3);
    }
    return v4i{(int)plane_place(d0, g0 + 0), (int)plane_place(d1, g0 + 1),
               (int)plane_place(d2, g0 + 2), (int)plane_place(d3, g0 + 3)};
}

// ------------------------------------------------------------------ staging

// Where this thread's chunks of a K tile live.  Thread tid owns chunks
// id = tid + i*NT: row id / CPR, 16-byte column id % CPR of the tile.  In
// the ALIGNED path (K % 16 == 0, 16-byte aligned operands) a chunk's buffer
// offset is fixed per tile and advanced by the K step; rows past M (N)
// carry kOOB and read zero.  Weight chunks at or past the end of the K range
// read zero as well, so the MFMAs of a ragged last K tile need no masking
// (the activation bytes there meet zero weights).
template <class C, bool ALIGNED, int KIND, bool PLANES>
struct Plan {
    rsrc_t rX, rW;
    uint32_t offA[C::A_LOADS];   // linear: byte offset at k = kb; conv: pixel base
    uint32_t offB[C::B_LOADS];
    int hA[C::A_LOADS], wA[C::A_LOADS];   // conv: pixel coordinates
    int kend;                             // end of the K range (bytes)

    __device__ __forceinline__ void init(const LayerDesc &d, int m0, int n0, int kb, int ke,
                                         int tid)
    {
        kend = ke;
        if constexpr (ALIGNED) {
            if constexpr (KIND == KIND_CONV3X3)
                rX = make_rsrc(d.X, (uint32_t)d.H * (uint32_t)d.Wd * (uint32_t)d.C);
            else
                rX = make_rsrc(d.X, (uint32_t)d.M * (uint32_t)d.K);
#pragma unroll
            for (int i = 0; i < C::A_LOADS; ++i) {
                const int id = tid + i * C::NT;
                const int m = m0 + id / C::CPR, c = id % C::CPR;
                if constexpr (KIND == KIND_CONV3X3) {
                    const bool ok = m < d.M;
                    const int h = ok ? m / d.Wd : -(1 << 20);
                    const int w = ok ? m - (m / d.Wd) * d.Wd : -(1 << 20);
                    hA[i] = h;
                    wA[i] = w;
                    offA[i] = ok ? (uint32_t)((h * d.Wd + w) * d.C) : 0u;
                } else {
                    offA[i] = m < d.M ? (uint32_t)m * (uint32_t)d.K + (uint32_t)(kb + 16 * c)
                                      : kOOB;
                }
            }
            if constexpr (!PLANES) {
                rW = make_rsrc(d.W, (uint32_t)d.N * (uint32_t)d.K);
#pragma unroll
                for (int i = 0; i < C::B_LOADS; ++i) {
                    const int id = tid + i * C::NT;
                    const int n = n0 + id / C::CPR, c = id % C::CPR;
                    offB[i] = n < d.N ? (uint32_t)n * (uint32_t)d.K + (uint32_t)(kb + 16 * c)
                                      : kOOB;
                }
            }
        }
    }

    // Implicit-GEMM chunk for C % 16 == 0: the chunk lies in one tap
    // (r, s); out-of-image taps, pixels past M and columns past K read zero.
    // When C is a multiple of BK the whole K tile lies in one tap, found once
    // (uniform) from the tile start k0.
    __device__ __forceinline__ v4i conv_chunk(const LayerDesc &d, int i, int k0, int c) const
    {
        const int kbyte = k0 + 16 * c;
        if (kbyte >= d.K)
            return zero4();
        int tap, ci;
        if (d.C % C::BK == 0) {
            tap = k0 / d.C;
            ci = k0 - tap * d.C + 16 * c;
        } else {
            tap = kbyte / d.C;
            ci = kbyte - tap * d.C;
        }
        const int r = tap / 3, s = tap - 3 * (tap / 3);
        const int hh = hA[i] + r - 1, ww = wA[i] + s - 1;
        const bool ok = (unsigned)hh < (unsigned)d.H && (unsigned)ww < (unsigned)d.Wd;
        const int delta = ((r - 1) * d.Wd + (s - 1)) * d.C + ci;
        return ld16(rX, ok ? (uint32_t)((int)offA[i] + delta) : kOOB);
    }
};

// One K tile of both operands held in registers between its global load and
// its LDS store.
template <class C, bool ALIGNED, int KIND, bool PLANES>
struct Regs {
    v4i a[C::A_LOADS];
    v4i b[C::B_LOADS];

    // Loads the K tile at absolute byte k0 = kb + kt.
    __device__ __forceinline__ void load(const Plan<C, ALIGNED, KIND, PLANES> &p,
                                         const LayerDesc &d, int m0, int n0, int k0, uint32_t kt,
                                         int tid)
    {
#pragma unroll
        for (int i = 0; i < C::A_LOADS; ++i) {
            const int id = tid + i * C::NT;
            const int r = id / C::CPR, c = id % C::CPR;
            if constexpr (!ALIGNED) {
                if constexpr (KIND == KIND_CONV3X3)
                    a[i] = load_conv_any(d, m0 + r, k0 + 16 * c);
                else
                    a[i] = load_rowmajor_any(d.X, d.M, d.K, m0 + r, k0 + 16 * c);
            } else if constexpr (KIND == KIND_CONV3X3) {
                a[i] = p.conv_chunk(d, i, k0, c);
            } else {
                a[i] = ld16(p.rX, p.offA[i] + kt);
            }
        }
#pragma unroll
        for (int i = 0; i < C::B_LOADS; ++i) {
            const int id = tid + i * C::NT;
            const int r = id / C::CPR, c = id % C::CPR;
            if constexpr (PLANES)
                b[i] = load_planes(d.P, d.N, d.K, d.bits, n0 + r, k0 + 16 * c);
            else if constexpr (!ALIGNED)
                b[i] = load_rowmajor_any(d.W, d.N, d.K, n0 + r, k0 + 16 * c);
            else
                b[i] = ld16(p.rW, k0 + 16 * c < p.kend ? p.offB[i] + kt : kOOB);
        }
    }

    __device__ __forceinline__ void store(v4i *sA, v4i *sB, uint32_t wmask, int tid) const
    {
        const int msk = (int)wmask;
#pragma unroll
        for (int i = 0; i < C::A_LOADS; ++i) {
            const int id = tid + i * C::NT;
            const int r = id / C::CPR, c = id % C::CPR;
            sA[r * C::CPR + swz<C::CPR>(r, c)] = a[i];
        }
#pragma unroll
        for (int i = 0; i < C::B_LOADS; ++i) {
            const int id = tid + i * C::NT;
            const int r = id / C::CPR, c = id % C::CPR;
            v4i v = b[i];
            if constexpr (!PLANES) {
                v.x &= msk;
                v.y &= msk;
                v.z &= msk;
                v.w &= msk;
            }
            sB[r * C::CPR + swz<C::CPR>(r, c)] = v;
        }
    }
};

// Accumulates the K range [kb, ke) of tile (m0, n0) into acc, two LDS stages.
//
// K tile t lives in LDS stage t % 2 while tile t+1 is written into the other
// stage and tiles t+2 .. t+PF are in flight in the register ring.  Within
// tile t, the LDS reads of sub-step kk+1 are in flight while the MFMAs of
// sub-step kk issue, one read after each MFMA (a run of reads can fill the
// LDS queue, and a wave that waits to issue a read issues no MFMA either).
// The one barrier per K tile sits before the last sub-step: by then every
// wave has read all of tile t's fragments and written its share of tile
// t+1, so the last sub-step's MFMAs (operands already in registers) cover
// the barrier and the reads of tile t+1's first fragments.  Tile t+1 is
// stored from the ring in the sub-step before the barrier (measured faster
// than half-way through tile t) and the ring slot is refilled right away,
// so a global load has PF whole K tiles to land.
//
// kloop is the loop proper: on entry tile 0 is in LDS stage 0 (visible to
// every wave) and tiles 1 .. PF are in the ring; mainloop adds the prologue
// that puts them there.
template <class C, bool ALIGNED, int KIND, bool PLANES>
__device__ __forceinline__ void kloop(const LayerDesc &d, uint32_t wmask, int m0, int n0, int kb,
                                      int nk, const Plan<C, ALIGNED, KIND, PLANES> &plan,
                                      Regs<C, ALIGNED, KIND, PLANES> (&ring)[C::PF],
                                      v16i (&acc)[C::FM][C::FN], v4i *smA, v4i *smB)
{
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
    constexpr int SA = C::BM * C::CPR, SB = C::BN * C::CPR;
    constexpr int KK = C::BK / 32;
    constexpr int WRITE_KK = KK - 2;          // sub-step that stores tile t+1
    constexpr int NW = C::A_LOADS + C::B_LOADS;

    v4i fa[2][C::FM], fb[2][C::FN];
    auto read = [&](int stage, int kk, v4i (&a)[C::FM], v4i (&b)[C::FN]) {
        const v4i *A = smA + stage * SA;
        const v4i *B = smB + stage * SB;
        const int c = 2 * kk + (lane >> 5);
#pragma unroll
        for (int i = 0; i < C::FM; ++i) {
            const int r = wm * C::WTM + i * 32 + (lane & 31);
            a[i] = A[r * C::CPR + swz<C::CPR>(r, c)];
        }
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
            const int r = wn * C::WTN + j * 32 + (lane & 31);
            b[j] = B[r * C::CPR + swz<C::CPR>(r, c)];
        }
    };
    auto mfmas = [&](v4i (&a)[C::FM], v4i (&b)[C::FN]) {
#pragma unroll
        for (int i = 0; i < C::FM; ++i)
#pragma unroll
            for (int j = 0; j < C::FN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[i], b[j], acc[i][j], 0, 0, 0);
    };

    read(0, 0, fa[0], fb[0]);
    int stage = 0;
    for (int t0 = 0; t0 < nk - 1; t0 += C::PF) {
#pragma unroll
        for (int u = 0; u < C::PF; ++u) {
            const int t = t0 + u;
            if (t < nk - 1) {
#pragma unroll
                for (int kk = 0; kk + 1 < KK; ++kk) {
                    read(stage, kk + 1, fa[(kk + 1) & 1], fb[(kk + 1) & 1]);
                    mfmas(fa[kk & 1], fb[kk & 1]);
                    if (kk == WRITE_KK) {
                        ring[u].store(smA + (stage ^ 1) * SA, smB + (stage ^ 1) * SB, wmask, tid);
                        if (t + 1 + C::PF < nk) {
                            const uint32_t off = (uint32_t)(t + 1 + C::PF) * C::BK;
                            ring[u].load(plan, d, m0, n0, kb + (int)off, off, tid);
                        }
#pragma unroll
                        for (int i = 0; i < C::FM * C::FN; ++i) {
                            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                            if (i < C::FM + C::FN)
                                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                            if (i < NW)
                                __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
                        }
                    } else {
#pragma unroll
                        for (int i = 0; i < C::FM * C::FN; ++i) {
                            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                            if (i < C::FM + C::FN)
                                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                        }
                    }
                }
                __syncthreads();
                read(stage ^ 1, 0, fa[0], fb[0]);
                mfmas(fa[(KK - 1) & 1], fb[(KK - 1) & 1]);
#pragma unroll
                for (int i = 0; i < C::FM * C::FN; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    if (i < C::FM + C::FN)
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
            read(stage, kk + 1, fa[(kk + 1) & 1], fb[(kk + 1) & 1]);
        mfmas(fa[kk & 1], fb[kk & 1]);
        if (kk + 1 < KK)
            __builtin_amdgcn_sched_group_barrier(0x100, C::FM + C::FN, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, C::FM * C::FN, 0);
    }
}

template <class C>
__device__ __forceinline__ void zero_acc(v16i (&acc)[C::FM][C::FN])
{
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
            acc[i][j] = v16i{};
}

template <class C, bool ALIGNED, int KIND, bool PLANES = false>
__device__ __forceinline__ void mainloop(const LayerDesc &d, uint32_t wmask, int m0, int n0,
                                         int kb, int ke, v16i (&acc)[C::FM][C::FN], v4i *smA,
                                         v4i *smB)
{
    const int tid = threadIdx.x;
    zero_acc<C>(acc);
    const int nk = (ke - kb + C::BK - 1) / C::BK;
    if (nk <= 0)
        return;

    Plan<C, ALIGNED, KIND, PLANES> plan;
    plan.init(d, m0, n0, kb, ke, tid);
    Regs<C, ALIGNED, KIND, PLANES> ring[C::PF];

    // Prologue: tile 0 into stage 0, tiles 1 .. PF into the ring.
    ring[0].load(plan, d, m0, n0, kb, 0u, tid);
    ring[0].store(smA, smB, wmask, tid);
#pragma unroll
    for (int u = 0; u < C::PF; ++u)
        if (1 + u < nk)
            ring[u].load(plan, d, m0, n0, kb + (1 + u) * C::BK, (uint32_t)(1 + u) * C::BK, tid);
    __syncthreads();
    kloop<C, ALIGNED, KIND, PLANES>(d, wmask, m0, n0, kb, nk, plan, ring, acc, smA, smB);
}

// ------------------------------------------------------ low-rank branch

// fp32 t as hi + lo bfloat16 bit patterns: hi keeps the top 16 bits (an
// exact truncation), lo is the remainder t - hi (exact in fp32) rounded to
// nearest even, so hi + lo = t within 2^-16 |t|.
__device__ __forceinline__ void split_bf16(float t, uint32_t &hi, uint32_t &lo)
{
    const uint32_t u = __float_as_uint(t);
    hi = u >> 16;
    const uint32_t rem = __float_as_uint(t - __uint_as_float(u & 0xffff0000u));
    lo = (rem + 0x7fffu + ((rem >> 16) & 1u)) >> 16;
}

// Stages the tile's low-rank operands in LDS: T rows m0.. (fp32 [M][r],
// split into bfloat16 hi and lo parts) and U rows n0.. (bfloat16 [N][r]).
// Rows past M or N read zero through the buffer bounds.
template <class C>
__device__ __forceinline__ void stage_lowrank(const LayerDesc &d, int m0, int n0, char *lds)
{
    const int r = d.lr_r;
    const rsrc_t rU = make_rsrc(d.lr_U, (uint32_t)d.N * (uint32_t)r * 2u);
    char *Thi = lds, *Tlo = lds + C::BM * kLrPitch, *Us = lds + 2 * C::BM * kLrPitch;
    const int tpr = r / 4;
    for (int e = threadIdx.x; e < C::BM * tpr; e += C::NT) {
        const int row = e / tpr, c = e % tpr;
        // A plain float4 load: the components of a 16-byte buffer load taken
        // apart one by one here compiled to one dword load used four times.
        float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
        if (m0 + row < d.M)
            t = *reinterpret_cast<const float4 *>(d.lr_T + (size_t)(m0 + row) * r + 4 * c);
        uint32_t h[4], l[4];
        split_bf16(t.x, h[0], l[0]);
        split_bf16(t.y, h[1], l[1]);
        split_bf16(t.z, h[2], l[2]);
        split_bf16(t.w, h[3], l[3]);
        *reinterpret_cast<uint2 *>(Thi + row * kLrPitch + 8 * c) =
            make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
        *reinterpret_cast<uint2 *>(Tlo + row * kLrPitch + 8 * c) =
            make_uint2(l[0] | (l[1] << 16), l[2] | (l[3] << 16));
    }
    const int upr = r / 8;
    for (int e = threadIdx.x; e < C::BN * upr; e += C::NT) {
        const int row = e / upr, c = e % upr;
        *reinterpret_cast<v4i *>(Us + row * kLrPitch + 16 * c) =
            ld16(rU, ((uint32_t)(n0 + row) * (uint32_t)r + 8u * c) * 2u);
    }
}

// Stages, per tile row m, the activation sum that multiplies a weight zero
// point: R[m] = sum_k x_code[m][k] (+ K (128 - z_x) for asymmetric codes,
// whose x_hat carries the offset 128 - z_x in every element).
template <class C>
__device__ __forceinline__ void stage_rowsums(const LayerDesc &d, int m0, char *lds)
{
    float *R = reinterpret_cast<float *>(lds + (2 * C::BM + C::BN) * kLrPitch);
    const float off = d.act ? (float)d.K * (128.0f - d.act[1]) : 0.0f;
    for (int e = threadIdx.x; e < C::BM; e += C::NT)
        R[e] = m0 + e < d.M ? (float)d.xrs[m0 + e] + off : 0.0f;
}

// Adds f * R[row] to the 16 registers of a lane in a 32x32 block starting
// at tile row rl (register v: row rl + 8*(v/4) + 4*(l/32) + v%4): four
// 16-byte LDS reads.
template <class C>
__device__ __forceinline__ void add_rowsum_block(const char *lds, int rl, int lane, float f,
                                                 v16f &out)
{
    const float *R = reinterpret_cast<const float *>(lds + (2 * C::BM + C::BN) * kLrPitch);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const float4 t = *reinterpret_cast<const float4 *>(R + rl + 8 * q + 4 * (lane >> 5));
        out[4 * q + 0] += f * t.x;
        out[4 * q + 1] += f * t.y;
        out[4 * q + 2] += f * t.z;
        out[4 * q + 3] += f * t.w;
    }
}

// The 32x32 block (rows rl.., columns cl.. of the tile) of T U^T from the
// staged operands: per 16-wide step of the rank, one bfloat16 MFMA on the hi
// and one on the lo part of T, accumulated in fp32.  Same register layout
// as the integer accumulators.
template <class C>
__device__ __forceinline__ v16f lowrank_block(const char *lds, int r, int rl, int cl, int lane)
{
    const char *Thi = lds, *Tlo = lds + C::BM * kLrPitch, *Us = lds + 2 * C::BM * kLrPitch;
    const int ao = (rl + (lane & 31)) * kLrPitch + 16 * (lane >> 5);
    const int bo = (cl + (lane & 31)) * kLrPitch + 16 * (lane >> 5);
    v16f out = {};
#pragma unroll
    for (int s = 0; s < kLowrankMaxRank / 16; ++s) {
        if (16 * s < r) {
            const v8bf b = __builtin_bit_cast(v8bf, *reinterpret_cast<const v4i *>(Us + bo + 32 * s));
            const v8bf ah = __builtin_bit_cast(v8bf, *reinterpret_cast<const v4i *>(Thi + ao + 32 * s));
            const v8bf al = __builtin_bit_cast(v8bf, *reinterpret_cast<const v4i *>(Tlo + ao + 32 * s));
            out = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, b, out, 0, 0, 0);
            out = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, b, out, 0, 0, 0);
        }
    }
    return out;
}

// Writes a finished tile: int32 accumulators and/or the fp32 dequantised
// value y = float(acc) * (sx * sw[n]) + bias[n].  With asymmetric
// activations (d.act) the zero point enters through the channel sum of W_b:
// y = (float(acc) + (128 - z) * colsum_b[n]) * (alpha * sw[n]) + bias[n].
// With a low-rank branch (d.lr_T) y also gains (T U^T)[m][n], and with
// per-channel weight zero points (d.wz: w_hat = sw (W_b + 128 - z_n)) the
// term (128 - z_n) R[m] joins the accumulator, R[m] the row's activation
// sum; both are computed from operands staged in the (then idle) LDS.  Register v of a 32x32
// accumulator in lane l is row 8*(v/4) + 4*(l/32) + v%4, column l%32, so
// each store instruction covers two 128-byte row segments.  Rows past M
// fall past the buffer end and are dropped; columns past N carry kOOB.
//
// Three parts, so that a persistent kernel can issue the next tile's loads
// after every read of the epilogue and before its stores: epilogue_stage
// (the LDS operands, called by every wave), epilogue_cols (the per-column
// factors of this lane) and epilogue_write (the stores).
template <class C>
struct EpiCols {
    float scale[C::FN], bias[C::FN], corr[C::FN], wsc[C::FN];
    uint32_t base[C::FN];   // byte offset of (row mrow, column n), kOOB past N
};

template <class C>
__device__ __forceinline__ void epilogue_stage(const LayerDesc &d, int m0, int n0, char *lds)
{
    const bool lowrank = d.lr_T != nullptr && d.y != nullptr;
    const bool wzero = d.wz != nullptr && d.y != nullptr;
    if (lowrank || wzero) {
        __syncthreads();            // every wave is done with the main loop's LDS
        if (lowrank)
            stage_lowrank<C>(d, m0, n0, lds);
        if (wzero)
            stage_rowsums<C>(d, m0, lds);
        __syncthreads();
    }
}

template <class C>
__device__ __forceinline__ void epilogue_cols(const LayerDesc &d, int m0, int n0, int bits,
                                              EpiCols<C> &ec)
{
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
    const bool wzero = d.wz != nullptr && d.y != nullptr;
    const int mrow = m0 + wm * C::WTM + 4 * (lane >> 5);
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
        const int n = n0 + wn * C::WTN + j * 32 + (lane & 31);
        const bool nok = n < d.N;
        float scale = 0.f, bias = 0.f, corr = 0.f, wsc = 0.f;
        if (nok) {
            if (d.act) {
                scale = d.act[0] * d.sw[n];
                corr = (128.0f - d.act[1]) * (float)d.colsums[(bits - 1) * d.N + n];
            } else {
                scale = d.sx * d.sw[n];
            }
            if (d.bias)
                bias = d.bias[n];
            if (wzero)
                wsc = (128.0f - d.wz[n]) * scale;
        }
        ec.scale[j] = scale;
        ec.bias[j] = bias;
        ec.corr[j] = corr;
        ec.wsc[j] = wsc;
        ec.base[j] = nok ? ((uint32_t)mrow * (uint32_t)d.N + (uint32_t)n) * 4u : kOOB;
    }
}

// EXTRAS = false compiles out the low-rank and weight-zero-point terms (the
// caller guarantees that no layer has them).
template <class C, bool NT = true, bool EXTRAS = true, int J0 = 0, int J1 = C::FN>
__device__ __forceinline__ void epilogue_write(const LayerDesc &d,
                                               const v16i (&acc)[C::FM][C::FN],
                                               const EpiCols<C> &ec, const char *lds)
{
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
    const bool lowrank = EXTRAS && d.lr_T != nullptr && d.y != nullptr;
    const bool wzero = EXTRAS && d.wz != nullptr && d.y != nullptr;
    const uint32_t outb = (uint32_t)d.M * (uint32_t)d.N * 4u;
    const rsrc_t ry = make_rsrc(d.y, d.y ? outb : 0u);
    const rsrc_t ra = make_rsrc(d.acc, d.acc ? outb : 0u);
    const uint32_t rowb = (uint32_t)d.N * 4u;
#pragma unroll
    for (int j = J0; j < J1; ++j) {
        const float scale = ec.scale[j], bias = ec.bias[j], corr = ec.corr[j], wsc = ec.wsc[j];
        const uint32_t base = ec.base[j];
        if (d.acc) {
#pragma unroll
            for (int i = 0; i < C::FM; ++i)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    if constexpr (NT)
                        st32(ra, base + (uint32_t)(i * 32 + 8 * (v >> 2) + (v & 3)) * rowb,
                             (uint32_t)acc[i][j][v]);
                    else
                        st32_cached(ra, base + (uint32_t)(i * 32 + 8 * (v >> 2) + (v & 3)) * rowb,
                                    (uint32_t)acc[i][j][v]);
        }
        if (d.y) {
#pragma unroll
            for (int i = 0; i < C::FM; ++i) {
                if (lowrank || wzero) {
                    v16f extra = {};
                    if (lowrank)
                        extra = lowrank_block<C>(lds, d.lr_r, wm * C::WTM + i * 32,
                                                 wn * C::WTN + j * 32, lane);
                    if (wzero)
                        add_rowsum_block<C>(lds, wm * C::WTM + i * 32, lane, wsc, extra);
#pragma unroll
                    for (int v = 0; v < 16; ++v)
                        st32(ry, base + (uint32_t)(i * 32 + 8 * (v >> 2) + (v & 3)) * rowb,
                             __builtin_bit_cast(uint32_t, ((float)acc[i][j][v] + corr) * scale +
                                                              bias + extra[v]));
                } else {
#pragma unroll
                    for (int v = 0; v < 16; ++v)
                        st32(ry, base + (uint32_t)(i * 32 + 8 * (v >> 2) + (v & 3)) * rowb,
                             __builtin_bit_cast(uint32_t,
                                                ((float)acc[i][j][v] + corr) * scale + bias));
                }
            }
        }
    }
}

template <class C, bool NT = true>
__device__ __forceinline__ void epilogue(const LayerDesc &d, int m0, int n0,
                                         const v16i (&acc)[C::FM][C::FN], int bits, char *lds)
{
    epilogue_stage<C>(d, m0, n0, lds);
    EpiCols<C> ec;
    epilogue_cols<C>(d, m0, n0, bits, ec);
    epilogue_write<C, NT>(d, acc, ec, lds);
}

// Workgroups are dispatched round-robin over the 8 XCDs (workgroup i runs on
// XCD i % 8), each with its own L2.  This bijection of [0, G) gives every XCD
// one contiguous range of logical tiles, so neighbouring tiles -- which share
// activation rows and weight columns -- meet in the same L2.
__device__ __forceinline__ int xcd_remap(int pid, int G)
{
    constexpr int NX = 8;
    const int per = (G + NX - 1) / NX;
    int tall = G % NX;
    if (tall == 0)
        tall = NX;
    const int xcd = pid % NX, local = pid / NX;
    if (xcd < tall)
        return xcd * per + local;
    return tall * per + (xcd - tall) * (per - 1) + local;
}

// Tile order within a layer: groups of GROUP_M tile rows are walked column by
// column, so that consecutive tiles share weight tiles and activation rows.
__device__ __forceinline__ void tile_coords(int t, int tiles_m, int tiles_n, int &tm, int &tn)
{
    constexpr int GROUP_M = 8;
    const int per_group = GROUP_M * tiles_n;
    const int g = t / per_group;
    const int first_m = g * GROUP_M;
    const int gm = min(tiles_m - first_m, GROUP_M);
    const int in = t - g * per_group;
    tm = first_m + in % gm;
    tn = in / gm;
}

template <class C, bool ALIGNED, int KIND, bool PLANES>
__global__ void __launch_bounds__(C::NT, C::OCC) k_masked_gemm(LayerDesc d)
{
    __shared__ v4i smA[C::SMA];
    __shared__ v4i smB[C::NSTAGE * C::BN * C::CPR];
    int tm, tn;
    tile_coords(xcd_remap(blockIdx.x, gridDim.x), d.tiles_m, d.tiles_n, tm, tn);
    const int m0 = tm * C::BM, n0 = tn * C::BN;
    v16i acc[C::FM][C::FN];
    mainloop<C, ALIGNED, KIND, PLANES>(d, keep_mask_dword(d.bits), m0, n0, 0, d.K, acc, smA,
                                       smB);
    epilogue<C>(d, m0, n0, acc, d.bits, reinterpret_cast<char *>(smA));
}

// Segment (run of one layer's tiles) of work unit t in a grouped launch:
// the last segment whose first unit is at or before t.
__device__ __forceinline__ int find_segment(const LayerDesc *__restrict__ descs, int L, int t)
{
    int lo = 0, hi = L - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (descs[mid].tile_begin <= t)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// Grouped launch over every layer of one denoising step: workgroup t finds
// its segment (a run of one layer's tiles) by binary search over the
// segments' first work units, and the layer's b from the (layer, stage)
// table (App. G.1: a table lookup, no re-launch).  CONV adds the
// implicit-GEMM path for 3x3 conv layers; without it every layer must be
// linear.
template <class C, bool CONV>
__global__ void __launch_bounds__(C::NT, C::OCC)
k_masked_gemm_grouped(const LayerDesc *__restrict__ descs, int L, const uint8_t *table, int S,
                      int stage)
{
    __shared__ v4i smA[C::SMA];
    __shared__ v4i smB[C::NSTAGE * C::BN * C::CPR];
    const int t = xcd_remap(blockIdx.x, gridDim.x);
    const LayerDesc d = descs[find_segment(descs, L, t)];
    const int bits = table[d.layer * S + stage];
    const uint32_t wmask = keep_mask_dword(bits);
    int tm, tn;
    tile_coords(t - d.tile_begin + d.tile_first, d.tiles_m, d.tiles_n, tm, tn);
    const int m0 = tm * C::BM, n0 = tn * C::BN;
    v16i acc[C::FM][C::FN];
    if (CONV && d.kind == KIND_CONV3X3)
        mainloop<C, true, KIND_CONV3X3>(d, wmask, m0, n0, 0, d.K, acc, smA, smB);
    else
        mainloop<C, true, KIND_LINEAR>(d, wmask, m0, n0, 0, d.K, acc, smA, smB);
    epilogue<C>(d, m0, n0, acc, bits, reinterpret_cast<char *>(smA));
}

// Persistent form of the grouped launch (linear layers, aligned operands,
// no low-rank branch and no weight zero points):
// one workgroup per compute unit walks the work units of its XCD's
// contiguous run, unit x*span + j, + wgs, + 2 wgs, ... (the same units a
// non-persistent launch would give that XCD, in the same order).  What it
// gains over one workgroup per tile is overlap at the tile boundary: the
// next tile's first K tile is loaded into registers between the two halves
// of the current tile's stores, so its latency is spent under the second
// half, and the stores (write-only, never waited for) drain while the next
// tile starts.  A vector-memory wait covers every older load and store, so
// those loads go out before the second half of the stores, not after all of
// them.
template <class C>
__device__ __forceinline__ void unit_coords(const LayerDesc &d, int t, int &m0, int &n0)
{
    int tm, tn;
    tile_coords(t - d.tile_begin + d.tile_first, d.tiles_m, d.tiles_n, tm, tn);
    m0 = tm * C::BM;
    n0 = tn * C::BN;
}

template <class C>
__global__ void __launch_bounds__(C::NT, C::OCC)
k_masked_gemm_persistent(const LayerDesc *__restrict__ descs, int L, int total, XcdRuns runs,
                         const uint8_t *__restrict__ table, int S, int stage, int parties)
{
    __shared__ v4i smA[C::SMA];
    __shared__ v4i smB[C::NSTAGE * C::BN * C::CPR];
    using PlanT = Plan<C, true, KIND_LINEAR, false>;
    using RegsT = Regs<C, true, KIND_LINEAR, false>;
    constexpr int NX = 8;
    const int tid = threadIdx.x;
    // The XCD's run of units is cut into `parties` contiguous parts, each
    // walked by wgs / parties of its workgroups (host: gridDim.x % 8 == 0,
    // wgs % parties == 0), so that one XCD works on several places of the
    // layer sequence at once.
    const int wgs = gridDim.x / NX / parties;       // workgroups per part
    const int x = blockIdx.x % NX, j = blockIdx.x / NX;
    const int part = j % parties, jj = j / parties;
    const int xbeg = runs.begin[x], xend = runs.begin[x + 1];
    const int pspan = (xend - xbeg + parties - 1) / parties;
    const int ubeg = xbeg + part * pspan;
    const int uend = min(xend, ubeg + pspan);
    int u = ubeg + jj;
    if (u >= uend)
        return;

    // The next tile's first K tile is loaded into ring slot 0, which is
    // free once a K loop has ended, and stored to LDS at the top of the
    // tile loop, where the slot is refilled with K tile 1 (the prologue of
    // mainloop, with its first load moved into the previous epilogue).
    PlanT plan;
    RegsT ring[C::PF];
    auto issue_first = [&](const LayerDesc &d, int m0, int n0) {
        // An opaque copy of the thread index: the chunk offsets are
        // recomputed here rather than kept live (or spilled) across the tile.
        int t = tid;
        asm volatile("" : "+v"(t));
        plan.init(d, m0, n0, 0, d.K, t);
        ring[0].load(plan, d, m0, n0, 0, 0u, t);
    };
    // b of a segment from the (layer, stage) table, read as an aligned
    // dword so that the uniform lookup is a scalar load (a vector load here
    // would wait for every store the wave has in flight).
    auto bits_of = [&](int sg) {
        const int idx = descs[sg].layer * S + stage;
        const uint32_t w = reinterpret_cast<const uint32_t *>(table)[idx >> 2];
        return (int)((w >> (8 * (idx & 3))) & 0xffu);
    };

    int seg = find_segment(descs, L, u);
    int m0, n0;
    unit_coords<C>(descs[seg], u, m0, n0);
    int bits = bits_of(seg);
    issue_first(descs[seg], m0, n0);
    for (;;) {
        const LayerDesc &d = descs[seg];
        const int nk = (d.K + C::BK - 1) / C::BK;
        const uint32_t wmask = keep_mask_dword(bits);
        __syncthreads();                            // no wave still reads the previous tile's LDS
        ring[0].store(smA, smB, wmask, tid);
        // Unconditional, so that no slot is live around the tile loop: a
        // tile past K reads zero weights through the buffer bounds and is
        // never consumed.
#pragma unroll
        for (int v = 0; v < C::PF; ++v)
            ring[v].load(plan, d, m0, n0, (1 + v) * C::BK, (uint32_t)(1 + v) * C::BK, tid);
        __syncthreads();
        v16i acc[C::FM][C::FN];
        zero_acc<C>(acc);
        kloop<C, true, KIND_LINEAR, false>(d, wmask, m0, n0, 0, nk, plan, ring, acc, smA, smB);
        const char *lds = reinterpret_cast<const char *>(smA);
        EpiCols<C> ec;
        epilogue_cols<C>(d, m0, n0, bits, ec);
        u += wgs;
        if (u >= uend) {
            epilogue_write<C, true, false>(d, acc, ec, lds);
            break;
        }
        // Another tile follows: the first half of the stores frees
        // accumulator registers, the next tile's first K tile is loaded,
        // and the second half of the stores covers the latency of those
        // loads.  (The ring slot they land in is dead after the K loop, so
        // no register set is live around the tile loop.)
        constexpr int JH = C::FN / 2;
        const LayerDesc &dp = d;
        seg = find_segment(descs, L, u);
        unit_coords<C>(descs[seg], u, m0, n0);
        bits = bits_of(seg);
        __builtin_amdgcn_sched_barrier(0);
        epilogue_write<C, true, false, 0, JH>(dp, acc, ec, lds);
        __builtin_amdgcn_sched_barrier(0);
        issue_first(descs[seg], m0, n0);
        __builtin_amdgcn_sched_barrier(0);
        epilogue_write<C, true, false, JH, C::FN>(dp, acc, ec, lds);
    }
}

// Split-K: work unit u holds tile u / splits and the K range of split
// sp = u % splits, [sp * kchunk, min(K, (sp + 1) * kchunk)) with kchunk a
// multiple of BK; its int32 partial tile goes to part + sp * M * N ([M][N]),
// summed in split order by k_split_finish.  The splits of one tile are
// consecutive units, so they run in one XCD and share its L2.
template <class C, int KIND>
__global__ void __launch_bounds__(C::NT, C::OCC)
k_masked_gemm_split(LayerDesc d, int32_t *part, int splits, int kchunk)
{
    __shared__ v4i smA[C::SMA];
    __shared__ v4i smB[C::NSTAGE * C::BN * C::CPR];
    const int u = xcd_remap(blockIdx.x, gridDim.x);
    const int t = u / splits, sp = u - t * splits;
    int tm, tn;
    tile_coords(t, d.tiles_m, d.tiles_n, tm, tn);
    const int m0 = tm * C::BM, n0 = tn * C::BN;
    const int k0 = sp * kchunk;
    const int k1 = min(d.K, k0 + kchunk);
    v16i acc[C::FM][C::FN];
    mainloop<C, true, KIND, false>(d, keep_mask_dword(d.bits), m0, n0, k0, k1, acc, smA, smB);
    LayerDesc dp = d;
    dp.acc = part + (size_t)sp * (size_t)d.M * (size_t)d.N;
    dp.y = nullptr;
    epilogue<C, false>(dp, m0, n0, acc, d.bits, reinterpret_cast<char *>(smA));
}

// ---------------------------------------------------------------- launchers

template <class C>
static void fill_tiles(LayerDesc &d)
{
    d.tiles_m = (d.M + C::BM - 1) / C::BM;
    d.tiles_n = (d.N + C::BN - 1) / C::BN;
}

template <class C>
hipError_t launch_single_cfg(const LayerDesc &din, bool aligned, hipStream_t stream)
{
    LayerDesc d = din;
    fill_tiles<C>(d);
    const long long grid = (long long)d.tiles_m * d.tiles_n;
    if (grid > 0x7fffffffLL)
        return hipErrorInvalidValue;
    dim3 g((unsigned)grid), b(C::NT);
    if (d.kind == KIND_CONV3X3) {
        if (aligned)
            hipLaunchKernelGGL((k_masked_gemm<C, true, KIND_CONV3X3, false>), g, b, 0, stream, d);
        else
            hipLaunchKernelGGL((k_masked_gemm<C, false, KIND_CONV3X3, false>), g, b, 0, stream,
                               d);
    } else if (aligned) {
        hipLaunchKernelGGL((k_masked_gemm<C, true, KIND_LINEAR, false>), g, b, 0, stream, d);
    } else {
        hipLaunchKernelGGL((k_masked_gemm<C, false, KIND_LINEAR, false>), g, b, 0, stream, d);
    }
    return hipGetLastError();
}

// Split-K partials of one aligned layer (see k_masked_gemm_split); the
// caller checks splits * M * N * 4 < 2^31 (32-bit buffer offsets).
template <class C>
hipError_t launch_split_cfg(const LayerDesc &din, int32_t *part, int splits, int kchunk,
                            hipStream_t stream)
{
    LayerDesc d = din;
    fill_tiles<C>(d);
    const long long grid = (long long)d.tiles_m * d.tiles_n * splits;
    if (grid > 0x7fffffffLL || splits < 1 || kchunk % C::BK != 0)
        return hipErrorInvalidValue;
    dim3 g((unsigned)grid), b(C::NT);
    if (d.kind == KIND_CONV3X3)
        hipLaunchKernelGGL((k_masked_gemm_split<C, KIND_CONV3X3>), g, b, 0, stream, d, part,
                           splits, kchunk);
    else
        hipLaunchKernelGGL((k_masked_gemm_split<C, KIND_LINEAR>), g, b, 0, stream, d, part,
                           splits, kchunk);
    return hipGetLastError();
}

template <class C>
hipError_t launch_planes_cfg(const LayerDesc &din, bool aligned, hipStream_t stream)
{
    LayerDesc d = din;
    fill_tiles<C>(d);
    const long long grid = (long long)d.tiles_m * d.tiles_n;
    if (grid > 0x7fffffffLL)
        return hipErrorInvalidValue;
    dim3 g((unsigned)grid), b(C::NT);
    if (aligned)
        hipLaunchKernelGGL((k_masked_gemm<C, true, KIND_LINEAR, true>), g, b, 0, stream, d);
    else
        hipLaunchKernelGGL((k_masked_gemm<C, false, KIND_LINEAR, true>), g, b, 0, stream, d);
    return hipGetLastError();
}

template <class C>
hipError_t launch_grouped_cfg(const LayerDesc *d_descs, int L, int total_tiles,
                              const uint8_t *d_table, int S, int stage, bool any_conv,
                              hipStream_t stream)
{
    dim3 g((unsigned)total_tiles), b(C::NT);
    if (any_conv)
        hipLaunchKernelGGL((k_masked_gemm_grouped<C, true>), g, b, 0, stream, d_descs, L, d_table,
                           S, stage);
    else
        hipLaunchKernelGGL((k_masked_gemm_grouped<C, false>), g, b, 0, stream, d_descs, L,
                           d_table, S, stage);
    return hipGetLastError();
}

// Persistent grouped launch over linear layers: wgs_per_xcd workgroups on
// each of the 8 XCDs.
template <class C>
hipError_t launch_persistent_cfg(const LayerDesc *d_descs, int L, int total_tiles,
                                 const XcdRuns &runs, const uint8_t *d_table, int S, int stage,
                                 int wgs_per_xcd, int parties, hipStream_t stream)
{
    if (wgs_per_xcd < 1 || total_tiles < 1 || parties < 1 || wgs_per_xcd % parties != 0 ||
        !xcd_runs_valid(runs, total_tiles))
        return hipErrorInvalidValue;
    dim3 g((unsigned)(8 * wgs_per_xcd)), b(C::NT);
    hipLaunchKernelGGL((k_masked_gemm_persistent<C>), g, b, 0, stream, d_descs, L, total_tiles,
                       runs, d_table, S, stage, parties);
    return hipGetLastError();
}

// Defines the dispatch entry of one tile configuration (a host function, so
// the table of host launchers never reaches the device compilation).
#define TASQ_DEFINE_TILE(NAME, CFG)                                                         \
    const TileOps &NAME()                                                                   \
    {                                                                                       \
        static const TileOps ops = {{CFG::BM, CFG::BN, CFG::BK}, &launch_single_cfg<CFG>,   \
                                    &launch_planes_cfg<CFG>, &launch_grouped_cfg<CFG>,      \
                                    &launch_split_cfg<CFG>, &launch_persistent_cfg<CFG>};   \
        return ops;                                                                         \
    }

}  // namespace tasq
