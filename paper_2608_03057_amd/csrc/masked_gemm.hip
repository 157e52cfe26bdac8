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
//   * global -> VGPR (16-byte loads, mask on the weight side) -> LDS, double
//     buffered with one barrier per K step, next tile's loads issued before
//     the current tile's MFMAs;
//   * LDS rows of BK bytes, 16-byte chunks XOR-swizzled so that the 32 rows
//     one MFMA operand read touches fall in distinct banks;
//   * each wave owns a (BM/WAVES_M) x (BN/WAVES_N) sub-tile of
//     v_mfma_i32_32x32x32_i8 accumulators (int32, exact);
//   * epilogue straight from the accumulators: lane l of a 32x32 block holds
//     column l%32, so every store instruction writes full 128-byte row
//     segments.
#include "tasq_internal.h"

namespace tasq {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

template <int BM_, int BN_, int BK_, int WAVES_M_, int WAVES_N_>
struct Cfg {
    static constexpr int BM = BM_, BN = BN_, BK = BK_;
    static constexpr int WAVES_M = WAVES_M_, WAVES_N = WAVES_N_;
    static constexpr int NT = WAVES_M * WAVES_N * 64;
    static constexpr int WTM = BM / WAVES_M, WTN = BN / WAVES_N;
    static constexpr int FM = WTM / 32, FN = WTN / 32;
    static constexpr int CPR = BK / 16;                 // 16-byte chunks per row
    static constexpr int A_LOADS = BM * CPR / NT;
    static constexpr int B_LOADS = BN * CPR / NT;
    static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile must hold 32x32 blocks");
    static_assert(BK % 32 == 0 && (CPR == 4 || CPR == 8), "BK must be 64 or 128");
    static_assert((BM * CPR) % NT == 0 && (BN * CPR) % NT == 0, "loads must divide");
};

using Cfg256x256 = Cfg<256, 256, 64, 2, 2>;
using Cfg128x256 = Cfg<128, 256, 128, 2, 2>;
using Cfg128x128 = Cfg<128, 128, 128, 2, 2>;
using Cfg64x64 = Cfg<64, 64, 128, 2, 2>;

TileShape tile_shape(int tile)
{
    switch (tile) {
    case TILE_256x256: return {256, 256, 64};
    case TILE_128x256: return {128, 256, 128};
    case TILE_128x128: return {128, 128, 128};
    default: return {64, 64, 128};
    }
}

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

// ---------------------------------------------------------------- loaders

__device__ __forceinline__ v4i zero4() { return v4i{0, 0, 0, 0}; }

// 16 bytes at p[0..15] with byte-wise bounds (K not a multiple of 16 or
// unaligned pointers); bytes with index >= valid read as zero.
__device__ __forceinline__ v4i load_bytes(const int8_t *p, int valid)
{
    uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < 16; ++i)
        if (i < valid)
            w[i >> 2] |= (uint32_t)(uint8_t)p[i] << (8 * (i & 3));
    return v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
}

// Chunk (row, kbyte..kbyte+15) of a row-major [rows][K] int8 matrix.
template <bool ALIGNED>
__device__ __forceinline__ v4i load_rowmajor(const int8_t *base, int rows, int K, int row,
                                             int kbyte)
{
    if (row >= rows || kbyte >= K)
        return zero4();
    const int8_t *p = base + (size_t)row * (size_t)K + kbyte;
    if constexpr (ALIGNED)
        return *reinterpret_cast<const v4i *>(p);
    else
        return load_bytes(p, K - kbyte);
}

// Chunk of the implicit-GEMM activation matrix of a 3x3 / pad 1 conv:
// row m = h*Wd + w, k = (r*3 + s)*C + ci -> X[h+r-1][w+s-1][ci] or 0.
// Needs C % 16 == 0 so a chunk never straddles two taps.
template <bool ALIGNED>
__device__ __forceinline__ v4i load_conv(const LayerDesc &d, int m, int kbyte)
{
    if (m >= d.M || kbyte >= d.K)
        return zero4();
    if constexpr (!ALIGNED) {
        // any C: each byte finds its own tap
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
    int tap = kbyte / d.C;
    int ci = kbyte - tap * d.C;
    int r = tap / 3, s = tap - 3 * (tap / 3);
    int h = m / d.Wd, w = m - (m / d.Wd) * d.Wd;
    int hh = h + r - 1, ww = w + s - 1;
    if (hh < 0 || hh >= d.H || ww < 0 || ww >= d.Wd)
        return zero4();
    const int8_t *p = d.X + ((size_t)hh * d.Wd + ww) * (size_t)d.C + ci;
    return *reinterpret_cast<const v4i *>(p);
}

// Bit i of x (i < 4) moved to bit 8*i: x * (1 + 2^7 + 2^14 + 2^21) places
// bit i at positions i + 7j, which are all distinct for i, j < 4, and only
// j = i lands on a multiple of 8.
__device__ __forceinline__ uint32_t spread4(uint32_t x)
{
    return (x * 0x00204081u) & 0x01010101u;
}

// Chunk (row n, kbyte..kbyte+15) of W_b rebuilt from the top b bit planes
// (App. G.2: the b-bit operand is the top b planes of the stored buffer;
// the dropped planes are never read).  Plane q contributes bit 7 - q of
// each byte; the result is the two's-complement byte of W_b.
__device__ __forceinline__ v4i load_planes(const uint32_t *P, int N, int K, int b, int n,
                                           int kbyte)
{
    if (n >= N || kbyte >= K)
        return zero4();
    const int KB = (K + 127) >> 7;
    const size_t plane_stride = (size_t)KB * (size_t)N * 4;
    const uint32_t *base = P + ((size_t)(kbyte >> 7) * N + n) * 4 + ((kbyte & 127) >> 5);
    const int sh = (kbyte & 16);
    uint32_t d0 = 0, d1 = 0, d2 = 0, d3 = 0;
    for (int q = 0; q < b; ++q) {
        const uint32_t half = base[q * plane_stride] >> sh;
        const int up = 7 - q;
        d0 |= spread4(half & 0xF) << up;
        d1 |= spread4((half >> 4) & 0xF) << up;
        d2 |= spread4((half >> 8) & 0xF) << up;
        d3 |= spread4((half >> 12) & 0xF) << up;
    }
    return v4i{(int)d0, (int)d1, (int)d2, (int)d3};
}

template <class C, bool ALIGNED, int KIND, bool PLANES>
struct Stage {
    v4i a[C::A_LOADS];
    v4i b[C::B_LOADS];

    __device__ __forceinline__ void load(const LayerDesc &d, int m0, int n0, int k0, int tid)
    {
#pragma unroll
        for (int i = 0; i < C::A_LOADS; ++i) {
            int id = tid + i * C::NT;
            int r = id / C::CPR, c = id % C::CPR;
            if constexpr (KIND == KIND_CONV3X3)
                a[i] = load_conv<ALIGNED>(d, m0 + r, k0 + 16 * c);
            else
                a[i] = load_rowmajor<ALIGNED>(d.X, d.M, d.K, m0 + r, k0 + 16 * c);
        }
#pragma unroll
        for (int i = 0; i < C::B_LOADS; ++i) {
            int id = tid + i * C::NT;
            int r = id / C::CPR, c = id % C::CPR;
            if constexpr (PLANES)
                b[i] = load_planes(d.P, d.N, d.K, d.bits, n0 + r, k0 + 16 * c);
            else
                b[i] = load_rowmajor<ALIGNED>(d.W, d.N, d.K, n0 + r, k0 + 16 * c);
        }
    }

    __device__ __forceinline__ void store(v4i *sA, v4i *sB, uint32_t wmask, int tid)
    {
        const int msk = (int)wmask;
#pragma unroll
        for (int i = 0; i < C::A_LOADS; ++i) {
            int id = tid + i * C::NT;
            int r = id / C::CPR, c = id % C::CPR;
            sA[r * C::CPR + swz<C::CPR>(r, c)] = a[i];
        }
#pragma unroll
        for (int i = 0; i < C::B_LOADS; ++i) {
            int id = tid + i * C::NT;
            int r = id / C::CPR, c = id % C::CPR;
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

// Accumulates the K range [kb, ke) of tile (m0, n0) into acc.
template <class C, bool ALIGNED, int KIND, bool PLANES = false>
__device__ __forceinline__ void mainloop(const LayerDesc &d, uint32_t wmask, int m0, int n0,
                                         int kb, int ke, v16i (&acc)[C::FM][C::FN],
                                         v4i *smA, v4i *smB)
{
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
    constexpr int SA = C::BM * C::CPR, SB = C::BN * C::CPR;

#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
            acc[i][j] = v16i{};

    const int nk = (ke - kb + C::BK - 1) / C::BK;
    if (nk <= 0)
        return;

    Stage<C, ALIGNED, KIND, PLANES> st;
    st.load(d, m0, n0, kb, tid);
    st.store(smA, smB, wmask, tid);
    __syncthreads();

    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        const bool more = kt + 1 < nk;
        if (more)
            st.load(d, m0, n0, kb + (kt + 1) * C::BK, tid);

        const v4i *A = smA + cur * SA;
        const v4i *B = smB + cur * SB;
#pragma unroll
        for (int kk = 0; kk < C::BK / 32; ++kk) {
            const int c = 2 * kk + (lane >> 5);
            v4i af[C::FM], bf[C::FN];
#pragma unroll
            for (int i = 0; i < C::FM; ++i) {
                int r = wm * C::WTM + i * 32 + (lane & 31);
                af[i] = A[r * C::CPR + swz<C::CPR>(r, c)];
            }
#pragma unroll
            for (int j = 0; j < C::FN; ++j) {
                int r = wn * C::WTN + j * 32 + (lane & 31);
                bf[j] = B[r * C::CPR + swz<C::CPR>(r, c)];
            }
#pragma unroll
            for (int i = 0; i < C::FM; ++i)
#pragma unroll
                for (int j = 0; j < C::FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[i], bf[j], acc[i][j],
                                                                      0, 0, 0);
        }
        if (more)
            st.store(smA + (cur ^ 1) * SA, smB + (cur ^ 1) * SB, wmask, tid);
        __syncthreads();
    }
}

// Writes a finished tile: int32 accumulators and/or the fp32 dequantised
// value.  Register v of a 32x32 accumulator in lane l is row
// 8*(v/4) + 4*(l/32) + v%4, column l%32.
template <class C>
__device__ __forceinline__ void epilogue(const LayerDesc &d, int m0, int n0,
                                         const v16i (&acc)[C::FM][C::FN])
{
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
        const int n = n0 + wn * C::WTN + j * 32 + (lane & 31);
        const bool nok = n < d.N;
        float scale = 0.f, bias = 0.f;
        if (nok) {
            scale = d.sx * d.sw[n];
            if (d.bias)
                bias = d.bias[n];
        }
#pragma unroll
        for (int i = 0; i < C::FM; ++i) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + wm * C::WTM + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                if (nok && m < d.M) {
                    const size_t o = (size_t)m * (size_t)d.N + n;
                    const int a = acc[i][j][v];
                    if (d.acc)
                        d.acc[o] = a;
                    if (d.y)
                        d.y[o] = (float)a * scale + bias;
                }
            }
        }
    }
}

// Tile order: groups of GROUP_M tile rows are walked column by column so
// that consecutive workgroups share weight tiles and activation rows in L2.
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
__global__ void __launch_bounds__(C::NT) k_masked_gemm(LayerDesc d)
{
    __shared__ v4i smA[2 * C::BM * C::CPR];
    __shared__ v4i smB[2 * C::BN * C::CPR];
    int tm, tn;
    tile_coords(blockIdx.x, d.tiles_m, d.tiles_n, tm, tn);
    const int m0 = tm * C::BM, n0 = tn * C::BN;
    v16i acc[C::FM][C::FN];
    mainloop<C, ALIGNED, KIND, PLANES>(d, keep_mask_dword(d.bits), m0, n0, 0, d.K, acc, smA,
                                       smB);
    epilogue<C>(d, m0, n0, acc);
}

// Grouped launch over every layer of one denoising step: workgroup t finds
// its layer by binary search over the tile prefix, and that layer's b from
// the (layer, stage) table (App. G.1: a table lookup, no re-launch).
template <class C>
__global__ void __launch_bounds__(C::NT)
k_masked_gemm_grouped(const LayerDesc *__restrict__ descs, int L, const uint8_t *table, int S,
                      int stage)
{
    __shared__ v4i smA[2 * C::BM * C::CPR];
    __shared__ v4i smB[2 * C::BN * C::CPR];
    const int t = blockIdx.x;
    int lo = 0, hi = L - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
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
    if (d.kind == KIND_CONV3X3)
        mainloop<C, true, KIND_CONV3X3>(d, wmask, m0, n0, 0, d.K, acc, smA, smB);
    else
        mainloop<C, true, KIND_LINEAR>(d, wmask, m0, n0, 0, d.K, acc, smA, smB);
    epilogue<C>(d, m0, n0, acc);
}

// ---------------------------------------------------------------- launchers

template <class C>
static hipError_t launch_single_cfg(const LayerDesc &din, bool aligned, hipStream_t stream)
{
    LayerDesc d = din;
    d.tiles_m = (d.M + C::BM - 1) / C::BM;
    d.tiles_n = (d.N + C::BN - 1) / C::BN;
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

template <class C>
static hipError_t launch_planes_cfg(const LayerDesc &din, bool aligned, hipStream_t stream)
{
    LayerDesc d = din;
    d.tiles_m = (d.M + C::BM - 1) / C::BM;
    d.tiles_n = (d.N + C::BN - 1) / C::BN;
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

hipError_t launch_bitplane(const LayerDesc &d, bool aligned, hipStream_t stream)
{
    return launch_planes_cfg<Cfg64x64>(d, aligned, stream);
}

hipError_t launch_single(const LayerDesc &d, int tile, bool aligned, void *ws,
                         hipStream_t stream)
{
    (void)ws;
    switch (tile) {
    case TILE_256x256: return launch_single_cfg<Cfg256x256>(d, aligned, stream);
    case TILE_128x256: return launch_single_cfg<Cfg128x256>(d, aligned, stream);
    case TILE_128x128: return launch_single_cfg<Cfg128x128>(d, aligned, stream);
    default: return launch_single_cfg<Cfg64x64>(d, aligned, stream);
    }
}

template <class C>
static hipError_t launch_grouped_cfg(const LayerDesc *d_descs, int L, int total_tiles,
                                     const uint8_t *d_table, int S, int stage,
                                     hipStream_t stream)
{
    dim3 g((unsigned)total_tiles), b(C::NT);
    hipLaunchKernelGGL((k_masked_gemm_grouped<C>), g, b, 0, stream, d_descs, L, d_table, S,
                       stage);
    return hipGetLastError();
}

hipError_t launch_grouped(const LayerDesc *d_descs, int L, int total_tiles,
                          const uint8_t *d_table, int S, int stage, int tile,
                          hipStream_t stream)
{
    switch (tile) {
    case TILE_256x256:
        return launch_grouped_cfg<Cfg256x256>(d_descs, L, total_tiles, d_table, S, stage, stream);
    case TILE_128x256:
        return launch_grouped_cfg<Cfg128x256>(d_descs, L, total_tiles, d_table, S, stage, stream);
    case TILE_128x128:
        return launch_grouped_cfg<Cfg128x128>(d_descs, L, total_tiles, d_table, S, stage, stream);
    default:
        return launch_grouped_cfg<Cfg64x64>(d_descs, L, total_tiles, d_table, S, stage, stream);
    }
}

size_t splitk_workspace_bytes(const LayerDesc &d, int tile)
{
    (void)d;
    (void)tile;
    return 0;
}

}  // namespace tasq
