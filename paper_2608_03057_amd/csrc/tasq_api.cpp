// C ABI of the TASQ masked quantized linear layer: argument validation,
// variant/tile choice, launches, schedule runner.  See include/tasq.h for the
// contract of every entry point.
#include "tasq.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "tasq_internal.h"

using tasq::LayerDesc;

namespace {

constexpr size_t kWsAlign = 256;

// XCDs of the device; the grouped GEMM kernels give each one a contiguous
// run of work units (xcd_remap in gemm_core.h).
constexpr int kXcds = 8;
constexpr int kComputeUnits = 256;
constexpr double kImbalanceLimit = 1.10;

// Cost of a 256x256 tile of the persistent step in bytes of K: its K plus a
// fixed part for its epilogue and the next tile's prologue.  The 28-block
// PixArt-shaped step (4.13 ms, 147 tiles per compute unit, 12.2 K tiles of
// 128 each on average) spends about 0.66 ms in tile ends, 4.5 us per tile,
// against 1.9 us per K tile: about 300 bytes of K.
constexpr double kTileFixedK = 384.0;

// The XCD runs of a persistent launch: contiguous in the work-unit order
// (neighbouring tiles share operands in one L2) and cut at about equal cost,
// a tile costing its K plus kTileFixedK.  Equal counts of tiles would give
// the XCD whose run ends a block later in the 28-block PixArt-shaped step
// (more 4608-deep tiles) 3% more work than the mean.
tasq::XcdRuns cost_runs(const std::vector<LayerDesc> &segs, long long total)
{
    double all = 0;
    for (const LayerDesc &d : segs)
        all += (double)d.tiles_m * d.tiles_n * ((double)d.K + kTileFixedK);
    tasq::XcdRuns r = {};
    int x = 1;
    double cum = 0;
    for (const LayerDesc &d : segs) {
        const long long n = (long long)d.tiles_m * d.tiles_n;
        const double c = (double)d.K + kTileFixedK;
        while (x < kXcds && cum + (double)n * c >= all * x / kXcds) {
            long long take = (long long)((all * x / kXcds - cum) / c + 0.5);
            take = take < 0 ? 0 : take > n ? n : take;
            r.begin[x] = (int)(d.tile_begin + take);
            ++x;
        }
        cum += (double)n * c;
    }
    for (; x < kXcds; ++x)
        r.begin[x] = (int)total;
    r.begin[kXcds] = (int)total;
    for (int i = 1; i <= kXcds; ++i)
        if (r.begin[i] < r.begin[i - 1])
            r.begin[i] = r.begin[i - 1];
    return r;
}

// Heaviest XCD run over the mean, for the per-layer tile order, a tile
// costing about its K plus a fixed part for loading and writing the tile.
double xcd_imbalance(const std::vector<LayerDesc> &descs, long long G)
{
    const long long per = (G + kXcds - 1) / kXcds;
    long long tall = G % kXcds;
    if (tall == 0)
        tall = kXcds;
    double work[kXcds] = {0};
    size_t l = 0;
    long long used = 0;          // tiles of layer l already assigned
    double total = 0;
    for (int x = 0; x < kXcds; ++x) {
        long long cnt = x < tall ? per : per - 1;
        while (cnt > 0 && l < descs.size()) {
            const long long n = (long long)descs[l].tiles_m * descs[l].tiles_n - used;
            const long long take = n < cnt ? n : cnt;
            const double w = (double)take * ((double)descs[l].K + 1024.0);
            work[x] += w;
            total += w;
            cnt -= take;
            used += take;
            if (used == (long long)descs[l].tiles_m * descs[l].tiles_n) {
                ++l;
                used = 0;
            }
        }
    }
    double mx = 0;
    for (double w : work)
        mx = w > mx ? w : mx;
    return total > 0 ? mx / (total / kXcds) : 1.0;
}

constexpr size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

int variant_of_opts(const tasq_opts *o) { return o ? o->variant : TASQ_VARIANT_AUTO; }

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_dims(long long M, long long N, long long K)
{
    if (M < 0 || N < 0 || K < 0)
        return TASQ_ERR_DIM;
    if (K > TASQ_MAX_K)
        return TASQ_ERR_OVERFLOW;
    return TASQ_OK;
}

// The variant value, split_k and the alignment of the optional buffers.
// Whether the layer has the weight copy its variant reads is checked per
// layer (check_weights).
int check_variant(const tasq_opts *o)
{
    const int v = variant_of_opts(o);
    if (v != TASQ_VARIANT_AUTO && v != TASQ_VARIANT_MASKED_I8 && v != TASQ_VARIANT_BITPLANE &&
        v != TASQ_VARIANT_PACKED)
        return TASQ_ERR_KIND;
    if (o && o->split_k < 0)
        return TASQ_ERR_RANGE;
    if (o && o->W_packed && !aligned16(o->W_packed))
        return TASQ_ERR_ALIGN;
    if (o && o->workspace && (reinterpret_cast<uintptr_t>(o->workspace) % kWsAlign) != 0)
        return TASQ_ERR_ALIGN;
    return TASQ_OK;
}

// Tuning overrides carried in tasq_opts (0 = the library's choice).
int forced_tile(const tasq_opts *o) { return o && o->tile > 0 ? o->tile - 1 : -1; }

int forced_ptile(const tasq_opts *o) { return o && o->packed_tile > 0 ? o->packed_tile - 1 : -1; }

int check_tuning(const tasq_opts *o)
{
    if (!o)
        return TASQ_OK;
    if (o->tile < 0 || o->tile > tasq::TILE_COUNT || o->packed_tile < 0 ||
        o->packed_tile > tasq::PTILE_COUNT || o->persistent < 0 || o->persistent > 2 ||
        o->persistent_wgs < 0 || o->persistent_wgs > 1024 || o->persistent_parties < 0 ||
        o->persistent_parties > 1024)
        return TASQ_ERR_RANGE;
    return TASQ_OK;
}

// The grouped step over linear layers without low-rank or weight-zero-point
// terms runs as a persistent launch (one workgroup per compute unit, tile
// boundaries overlapped) with the 256x256 tile once there are at least two
// tiles per compute unit, unless the caller forces it off or on.
bool use_persistent(const tasq_opts *o, bool big_tile, long long total)
{
    if (o && o->persistent)
        return o->persistent == 2;
    return big_tile && total >= 2LL * kComputeUnits;
}

int persistent_wgs_per_xcd(const tasq_opts *o)
{
    return o && o->persistent_wgs > 0 ? o->persistent_wgs : kComputeUnits / kXcds;
}

// Parts of each XCD's run walked side by side by the persistent launch;
// falls back to 1 when the requested count does not divide the workgroups
// per XCD.
int persistent_parties(const tasq_opts *o, int wgs_per_xcd)
{
    const int p = o && o->persistent_parties > 0 ? o->persistent_parties : 1;
    return wgs_per_xcd % p == 0 ? p : 1;
}

// Packed-weight tile of a single launch, from a sweep of every tile over the
// DiT/UNet layer shapes with the Infinity Cache flushed before each launch:
// the 256x256 tile once it gives at least 140 tiles (even half a wave of
// 256x256 tiles beats 2-3 waves of smaller ones from about there), the
// 4-wave 128x256 tile (two workgroups per CU) while it gives 200 tiles, and
// 64x64 tiles below that.
int pick_packed_tile(const tasq_opts *o, long long M, long long N, long long K)
{
    const int f = forced_ptile(o);
    if (f >= 0)
        return f;
    const long long t256 = ((M + 255) / 256) * ((N + 255) / 256);
    const long long t128x256 = ((M + 127) / 128) * ((N + 255) / 256);
    if (t256 >= 140 || M * N * K >= (1LL << 38))
        return tasq::PTILE_256x256_K128_W8;
    if (t128x256 >= 200)
        return tasq::PTILE_128x256_K128_W4;
    return tasq::PTILE_64x64_K128_W4;
}

// Packed-weight tile of the grouped per-step launch.
int pick_packed_grouped_tile(const tasq_opts *o)
{
    const int f = forced_ptile(o);
    return f >= 0 ? f : tasq::PTILE_256x256_K128_W8;
}

// Tile used for a single (non-grouped) launch, from the same sweep: 256x256
// tiles (8 waves, BK 128) from 140 tiles up, 128x128 tiles while they give
// 200 tiles, 64x64 tiles below that so that more workgroups cover the 256
// compute units.
int pick_tile(const tasq_opts *o, long long M, long long N)
{
    const int f = forced_tile(o);
    if (f >= 0)
        return f;
    const long long t256 = ((M + 255) / 256) * ((N + 255) / 256);
    const long long t128 = ((M + 127) / 128) * ((N + 127) / 128);
    if (t256 >= 140)
        return tasq::TILE_256x256_K128_W8_PF1;
    if (t128 >= 200)
        return tasq::TILE_128x128_K128_W4_PF2;
    return tasq::TILE_64x64_K128_W4_PF2;
}

// Split-K of single-layer calls with the row-major weight.  A layer with few
// output tiles and a long K leaves most of the chip idle while each
// workgroup walks all of K; cutting K into s ranges gives s times the
// workgroups, at the price of writing and re-reading s int32 partial
// outputs (summed in a fixed order, so the result is exact and identical).
// Measured on the DiT/UNet shapes (cache flushed before each launch), the
// partial traffic outweighs the gain unless K is long and the 256x256 tiles
// few: the SDXL-Turbo 3x3 conv (K = 11520, 20 tiles) runs 75 -> 44 us with
// 10 ranges, while K <= 5600 layers ran 0-3x slower split.
constexpr int kSplitMinChunk = 1024;     // at least this much K per split
constexpr int kSplitMinK = 8192;
constexpr int kSplitMaxTiles = 64;

int auto_splits(long long M, long long N, long long K)
{
    const long long t256 = ((M + 255) / 256) * ((N + 255) / 256);
    if (t256 > kSplitMaxTiles || t256 == 0 || K < kSplitMinK)
        return 1;
    long long s = kComputeUnits / t256;
    const long long smax = K / kSplitMinChunk;
    if (s > smax)
        s = smax;
    return s >= 2 ? (int)s : 1;
}

// K range per split (a multiple of 128, the largest BK) and the resulting
// number of non-empty splits.
void split_geometry(int K, int s, int &kchunk, int &splits)
{
    const int per = (K + s - 1) / s;
    kchunk = (per + 127) / 128 * 128;
    splits = (K + kchunk - 1) / kchunk;
}

// Split-K partials of the largest layer a schedule would split (0 when
// none would): the schedule workspace keeps room for them after the device
// layer list and the bit table.
size_t max_split_bytes(const tasq_layer *layers, int L)
{
    unsigned long long mx = 0;
    for (int l = 0; l < L; ++l) {
        const tasq_layer &t = layers[l];
        if (t.M <= 0 || t.N <= 0 || t.K <= 128)
            continue;
        const int s = auto_splits(t.M, t.N, t.K);
        if (s < 2)
            continue;
        int kchunk, splits;
        split_geometry(t.K, s, kchunk, splits);
        const unsigned long long need = 4ULL * splits * (unsigned long long)t.M * t.N;
        if (need < (1ULL << 31) && need > mx)
            mx = need;
    }
    return (size_t)mx;
}

constexpr size_t schedule_partials_offset(int L)
{
    return round_up((size_t)L * kXcds * sizeof(LayerDesc), kWsAlign) +
           round_up((size_t)L * 64, kWsAlign);
}

int pick_split_tile(const tasq_opts *o)
{
    const int f = forced_tile(o);
    return f >= 0 ? f : tasq::TILE_256x256_K128_W8_PF1;
}

// Tile of the grouped per-step launch: 256x256, unless one 256x256 tile of
// the longest-K layer costs more than a compute unit's even share of the
// whole step; then that tile alone sets the step time (the 3x3 conv of the
// SDXL-Turbo block: K = 11520 against 0.5 GOP per CU), and 128x128 tiles cut
// it by four (measured 0.230 -> 0.178 ms per step there, no change on the
// DiT blocks, which keep 256x256).
int pick_grouped_tile(const tasq_opts *o, const std::vector<LayerDesc> &descs)
{
    const int f = forced_tile(o);
    if (f >= 0)
        return f;
    double total = 0, longest = 0;
    for (const LayerDesc &d : descs) {
        total += 2.0 * d.M * (double)d.N * d.K;
        const double tile = 2.0 * 256 * 256 * (double)d.K;
        longest = tile > longest ? tile : longest;
    }
    return longest > total / kComputeUnits ? tasq::TILE_128x128_K128_W4_PF2
                                           : tasq::TILE_256x256_K128_W8_PF1;
}

bool use_bitplane(const tasq_opts *o) { return o && o->variant == TASQ_VARIANT_BITPLANE; }

// The buffer-offset fast path also needs each input below 2 GiB.
bool fits_buffers(const LayerDesc &d)
{
    const long long xb = d.kind == tasq::KIND_CONV3X3 ? (long long)d.H * d.Wd * d.C
                                                       : (long long)d.M * d.K;
    return xb < (1LL << 31) && (long long)d.N * d.K < (1LL << 31);
}

// The packed buffer is addressed with 32-bit offsets.
bool packed_fits(const LayerDesc &d)
{
    return tasq::packed_weight_bytes_host(d.N, d.K) < (1ULL << 31);
}

// The planes are addressed with 32-bit offsets by the weight-streaming kernel.
bool planes_fit(const LayerDesc &d)
{
    return tasq::planes_bytes_host(d.N, d.K) < (1ULL << 31);
}

// Activation operand on the 16-byte buffer fast path.
bool x_aligned(const LayerDesc &d)
{
    const int inner = d.kind == tasq::KIND_CONV3X3 ? d.C : d.K;
    return inner % 16 == 0 && aligned16(d.X) && fits_buffers(d);
}

// A linear layer that the weight-streaming kernels take: few tokens and
// 16-byte activation rows.
bool skinny_shape(const LayerDesc &d)
{
    return d.kind == tasq::KIND_LINEAR && d.M <= tasq::kSkinnyMaxM && x_aligned(d);
}

// Which stored copy of the weight a layer reads.
enum WeightSrc { SRC_NONE = 0, SRC_ROWS, SRC_PACKED, SRC_PLANES };

// The variant names the copy; AUTO picks by shape from what is present.
// With few tokens the layer is a weight stream whose time follows the
// bytes read, so AUTO reads the top b planes there (App. G.2: only the
// surviving planes are fetched).  Measured on the 112-layer PixArt-shaped
// schedule (ms per denoising step, TASQ table of mean 4.94 bits / static
// b = 8): at M = 16 planes 0.058 / 0.093, packed int8 0.095 / 0.095, int8
// rows 0.108 / 0.101; at M = 32 planes 0.088 / 0.117, packed 0.111 / 0.111;
// at M = 64 planes 0.152 / 0.169, packed 0.181 / 0.181.  The plane stream
// wins at every b below 8; at b = 8 it reads as many bytes as the int8 copy
// and the two streams are within 7% of each other either way, so there AUTO
// keeps the packed copy when one is given.  For M in the
// thousands the weights are a few percent of the traffic and rebuilding the
// bytes from planes per output tile costs more than it saves, so AUTO takes
// the int8 copies, and the bit-plane GEMM only when no other copy is given.
// Between the two int8 copies (both given):
//   * a single layer takes the packed copy when it has more than one
//     256x256 tile per two compute units, the rows otherwise.  Measured per
//     layer (us, b = 8, cold cache, rows / packed): PixArt QKV 8192x1152x3456
//     (448 tiles) 60.4 / 57.0, MLP-up (576) 82.6 / 78.0, MLP-down (160)
//     72.5 / 71.0, SANA GLU-up (704) 145.4 / 133.4; SDXL-Turbo A-QKV (128)
//     17.8 / 18.4, B-QKV (60) 17.9 / 21.6, B-ff-down (20) 30.6 / 33.9, the
//     3x3 conv (20) 69.4 / 71.5, 256x1152x1152 (5) 10.6 / 12.1;
//   * a schedule takes the rows, whose grouped step runs as the persistent
//     launch: 4.23 ms per denoising step of the 28-block PixArt-shaped
//     schedule against 4.59 ms for the grouped packed-weight launch.
// any_below8: the layer runs at some b below 8 (its b for a single call; any
// entry of its table row for a schedule).
WeightSrc weight_source(const LayerDesc &d, const tasq_opts *o, bool any_below8,
                        bool in_schedule)
{
    const bool rows = d.W != nullptr, packed = d.Wp != nullptr, planes = d.P != nullptr;
    switch (variant_of_opts(o)) {
    case TASQ_VARIANT_BITPLANE:
        return planes && d.kind == tasq::KIND_LINEAR ? SRC_PLANES : SRC_NONE;
    case TASQ_VARIANT_PACKED:
        return packed ? SRC_PACKED : SRC_NONE;
    case TASQ_VARIANT_MASKED_I8:
        return rows ? SRC_ROWS : SRC_NONE;
    default:
        break;
    }
    const bool linear = d.kind == tasq::KIND_LINEAR;
    if (planes && linear && skinny_shape(d) && planes_fit(d) && (any_below8 || !packed))
        return SRC_PLANES;
    if (packed && rows && !skinny_shape(d)) {
        if (in_schedule)
            return aligned16(d.W) ? SRC_ROWS : SRC_PACKED;
        const long long tiles = (long long)((d.M + 255) / 256) * ((d.N + 255) / 256);
        return tiles > kComputeUnits / 2 ? SRC_PACKED : SRC_ROWS;
    }
    if (packed)
        return SRC_PACKED;
    if (rows)
        return SRC_ROWS;
    if (planes && linear)
        return SRC_PLANES;
    return SRC_NONE;
}

// Weight-streaming path for skinny activations: linear layers with M <= 64
// and 16-byte activation rows, reading the weight copy `src`.  Returns false
// when that copy cannot be streamed.
bool skinny_source(const LayerDesc &d, WeightSrc src, tasq::SkinnyWeights &out)
{
    if (!skinny_shape(d))
        return false;
    switch (src) {
    case SRC_PLANES:
        out = tasq::SKINNY_PLANES;
        return planes_fit(d);
    case SRC_PACKED:
        out = tasq::SKINNY_PACKED;
        return packed_fits(d);
    case SRC_ROWS:
        out = tasq::SKINNY_ROWS;
        return aligned16(d.W);
    default:
        return false;
    }
}

int launch_layer(const LayerDesc &d, const tasq_opts *o, hipStream_t stream,
                 bool allow_split = false)
{
    if (d.M == 0 || d.N == 0)
        return TASQ_OK;
    hipError_t e;
    const WeightSrc wsrc = weight_source(d, o, d.bits < 8, false);
    tasq::SkinnyWeights src;
    if (skinny_source(d, wsrc, src)) {
        e = tasq::launch_skinny(d, src, stream);
        return e == hipSuccess ? TASQ_OK : TASQ_ERR_HIP;
    }
    if (wsrc == SRC_PACKED && packed_fits(d)) {
        e = tasq::packed_tile_ops(pick_packed_tile(o, d.M, d.N, d.K))
                .single(d, x_aligned(d), stream);
        return e == hipSuccess ? TASQ_OK : TASQ_ERR_HIP;
    }
    if (wsrc == SRC_PLANES) {
        e = tasq::tile_ops(tasq::TILE_64x64_K128_W4_PF2).planes(
            d, (d.K % 16) == 0 && aligned16(d.X) && fits_buffers(d), stream);
    } else {
        bool aligned;
        if (d.kind == tasq::KIND_CONV3X3)
            aligned = (d.C % 16) == 0 && aligned16(d.X) && aligned16(d.W);
        else
            aligned = (d.K % 16) == 0 && aligned16(d.X) && aligned16(d.W);
        aligned = aligned && fits_buffers(d);
        // Split-K: forced (split_k >= 2, needs the workspace) or chosen
        // (split_k == 0, only with a large enough workspace).
        const int req = o ? o->split_k : 0;
        int splits = 1, kchunk = 0;
        if (allow_split && req != 1 && d.K > 128) {
            const int s = req >= 2 ? req : auto_splits(d.M, d.N, d.K);
            if (s > 1) {
                split_geometry(d.K, s, kchunk, splits);
                const unsigned long long need = 4ULL * splits * (unsigned long long)d.M * d.N;
                const bool ws_ok = o && o->workspace && o->workspace_bytes >= need &&
                                   need < (1ULL << 31);
                if (!ws_ok && req >= 2)
                    return TASQ_ERR_WORKSPACE;
                if (!ws_ok || !aligned)
                    splits = 1;
            }
        }
        if (splits > 1) {
            int32_t *part = static_cast<int32_t *>(o->workspace);
            e = tasq::tile_ops(pick_split_tile(o)).split(d, part, splits, kchunk, stream);
            if (e == hipSuccess)
                e = tasq::launch_split_finish(d, part, splits, stream);
        } else {
            e = tasq::tile_ops(pick_tile(o, d.M, d.N)).single(d, aligned, stream);
        }
    }
    return e == hipSuccess ? TASQ_OK : TASQ_ERR_HIP;
}

LayerDesc make_desc(const tasq_layer &L, const tasq_opts *o)
{
    LayerDesc d;
    std::memset(&d, 0, sizeof d);
    d.X = L.X;
    d.W = L.W;
    d.P = L.W_planes ? L.W_planes : (o ? o->W_planes : nullptr);
    d.Wp = L.W_packed ? L.W_packed : (o ? o->W_packed : nullptr);
    d.act = L.act_params ? L.act_params : (o ? o->act_params : nullptr);
    d.colsums = L.colsums ? L.colsums : (o ? o->colsums : nullptr);
    d.wz = L.w_zero ? L.w_zero : (o ? o->w_zero : nullptr);
    d.xrs = L.w_zero ? L.x_rowsums : (o ? o->x_rowsums : nullptr);
    if (L.lowrank_T) {
        d.lr_T = L.lowrank_T;
        d.lr_U = L.lowrank_up;
        d.lr_r = L.lowrank_rank;
    } else if (o && o->lowrank_T) {
        d.lr_T = o->lowrank_T;
        d.lr_U = o->lowrank_up;
        d.lr_r = o->lowrank_rank;
    }
    d.sw = L.sw;
    d.bias = L.bias;
    d.acc = L.acc;
    d.y = L.y;
    d.sx = L.sx;
    d.M = L.M;
    d.N = L.N;
    d.K = L.K;
    d.kind = L.kind;
    d.H = L.H;
    d.Wd = L.Wd;
    d.C = L.C;
    return d;
}

// The layer has the weight copy its variant reads: the planes (BITPLANE),
// the packed buffer (PACKED), the rows (MASKED_I8), or under AUTO any copy
// that serves the layer kind (the planes serve linear layers only).  The
// named copy must be present even when the layer is empty.
int check_weights(const tasq_layer &L, const tasq_opts &o, bool needs_w)
{
    const int v = o.variant;
    if (v == TASQ_VARIANT_BITPLANE && !o.W_planes)
        return TASQ_ERR_LAYOUT;
    if (v == TASQ_VARIANT_PACKED && !o.W_packed)
        return TASQ_ERR_LAYOUT;
    if (!needs_w || v == TASQ_VARIANT_BITPLANE || v == TASQ_VARIANT_PACKED)
        return TASQ_OK;
    if (v == TASQ_VARIANT_MASKED_I8)
        return L.W ? TASQ_OK : TASQ_ERR_NULL;
    const bool planes_serve = o.W_planes && L.kind == TASQ_KIND_LINEAR;
    return L.W || o.W_packed || planes_serve ? TASQ_OK : TASQ_ERR_NULL;
}

// Validation shared by single calls and schedule layers.
int validate_layer(const tasq_layer &L, const tasq_opts *o)
{
    if (L.kind != TASQ_KIND_LINEAR && L.kind != TASQ_KIND_CONV3X3)
        return TASQ_ERR_KIND;
    // A pointer is required only where its array has elements.
    const bool has_out = L.M > 0 && L.N > 0;
    if (L.M > 0 && L.K > 0 && !L.X)
        return TASQ_ERR_NULL;
    if (has_out && !L.acc && !L.y)
        return TASQ_ERR_NULL;
    if (has_out && L.y && !L.sw)
        return TASQ_ERR_NULL;
    tasq_opts local = o ? *o : tasq_opts{};
    if (L.W_planes)
        local.W_planes = L.W_planes;
    if (L.W_packed)
        local.W_packed = L.W_packed;
    if (L.act_params)
        local.act_params = L.act_params;
    if (L.colsums)
        local.colsums = L.colsums;
    // Asymmetric activations need the channel sums for the zero point.
    if (has_out && L.y && local.act_params && !local.colsums)
        return TASQ_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(local.act_params) & 3) ||
        (reinterpret_cast<uintptr_t>(local.colsums) & 3))
        return TASQ_ERR_ALIGN;
    // Weight zero points: the layer's own fields, else the call's.
    if (L.w_zero) {
        local.w_zero = L.w_zero;
        local.x_rowsums = L.x_rowsums;
    }
    if (has_out && L.y && local.w_zero) {
        if (!local.x_rowsums)
            return TASQ_ERR_NULL;
        if ((reinterpret_cast<uintptr_t>(local.w_zero) & 3) ||
            (reinterpret_cast<uintptr_t>(local.x_rowsums) & 3))
            return TASQ_ERR_ALIGN;
        if (L.kind == TASQ_KIND_CONV3X3)
            return TASQ_ERR_LAYOUT;
    }
    // Low-rank branch: the layer's own fields, else the call's.
    if (L.lowrank_T) {
        local.lowrank_T = L.lowrank_T;
        local.lowrank_up = L.lowrank_up;
        local.lowrank_rank = L.lowrank_rank;
    }
    if (has_out && L.y && local.lowrank_T) {
        if (!local.lowrank_up)
            return TASQ_ERR_NULL;
        if (local.lowrank_rank != 16 && local.lowrank_rank != 32)
            return TASQ_ERR_DIM;
        if ((reinterpret_cast<uintptr_t>(local.lowrank_T) & 15) ||
            (reinterpret_cast<uintptr_t>(local.lowrank_up) & 15))
            return TASQ_ERR_ALIGN;
        if (L.kind == TASQ_KIND_CONV3X3)
            return TASQ_ERR_LAYOUT;
        // Staged through 32-bit buffer offsets, with a tile's rows past M.
        if (((long long)L.M + 256) * local.lowrank_rank * 4 >= (1LL << 31) ||
            ((long long)L.N + 256) * local.lowrank_rank * 2 >= (1LL << 31))
            return TASQ_ERR_DIM;
    }
    const bool needs_w = L.N > 0 && L.K > 0;
    if (int rc = check_variant(&local))
        return rc;
    if (int rc = check_weights(L, local, needs_w))
        return rc;
    if (L.kind == TASQ_KIND_CONV3X3) {
        if (L.H < 0 || L.Wd < 0 || L.C < 0 || L.N < 0)
            return TASQ_ERR_DIM;
        if ((long long)L.M != (long long)L.H * L.Wd || (long long)L.K != 9LL * L.C)
            return TASQ_ERR_DIM;
        if (use_bitplane(&local))
            return TASQ_ERR_LAYOUT;     // the bit-plane kernel covers linear layers
        // A padded tap holds code 0, which dequantises to alpha (128 - z), not
        // to zero: asymmetric codes would need a per-pixel zero-point term.
        if (local.act_params)
            return TASQ_ERR_LAYOUT;
    }
    if (int rc = check_dims(L.M, L.N, L.K))
        return rc;
    // Without the row-major copy the packed buffer must be addressable.
    if (local.W_packed && !L.W && !use_bitplane(&local) &&
        tasq::packed_weight_bytes_host(L.N, L.K) >= (1ULL << 31))
        return TASQ_ERR_DIM;
    // Outputs are written through 32-bit buffer offsets (see gemm_core.h).
    if (((long long)L.M + 256) * (long long)L.N * 4 >= (1LL << 31))
        return TASQ_ERR_DIM;
    return TASQ_OK;
}


// Device-side layer list and bit table of tasq_run_schedule_noalloc: one
// copy per GPU the library runs on, held until the process ends.  Host code
// never uses the name itself (a host-side stand-in, not a device address):
// static_scratch() looks the address up once per device with that device
// current, and only that pointer reaches kernels and copies.
constexpr size_t kStaticScratchBytes = schedule_partials_offset(TASQ_STATIC_MAX_LAYERS);
static_assert(kStaticScratchBytes == TASQ_STATIC_SCRATCH_BYTES,
              "TASQ_STATIC_SCRATCH_BYTES must match the layer-list layout");
__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

// Device address of this stream's GPU's scratch array.
int static_scratch(hipStream_t stream, void **out)
{
    int cur = 0, dev = 0;
    if (hipGetDevice(&cur) != hipSuccess)
        return TASQ_ERR_HIP;
    dev = cur;
    if (stream && hipStreamGetDevice(stream, &dev) != hipSuccess)
        return TASQ_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices)
        return TASQ_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        if (dev != cur && hipSetDevice(dev) != hipSuccess)
            return TASQ_ERR_HIP;
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (dev != cur && hipSetDevice(cur) != hipSuccess)
            return TASQ_ERR_HIP;
        if (e != hipSuccess || !p)
            return TASQ_ERR_HIP;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return TASQ_OK;
}

}  // namespace

extern "C" {

const char *tasq_status_string(int status)
{
    switch (status) {
    case TASQ_OK: return "ok";
    case TASQ_ERR_NULL: return "required pointer is NULL or no output requested";
    case TASQ_ERR_DIM: return "bad dimension";
    case TASQ_ERR_BITS: return "effective bits outside [1, 8]";
    case TASQ_ERR_OVERFLOW: return "K too large for exact int32 accumulation";
    case TASQ_ERR_RANGE: return "bad stage/step range or count, or a buffer shared by two jobs";
    case TASQ_ERR_LAYOUT: return "requested variant needs a weight layout that is absent";
    case TASQ_ERR_WORKSPACE:
        return "workspace missing or too small (noalloc schedule: more layers than its scratch holds)";
    case TASQ_ERR_HIP: return "HIP runtime or launch failure";
    case TASQ_ERR_KIND: return "unknown layer kind or variant";
    case TASQ_ERR_ALIGN: return "workspace not 256-byte aligned or packed weight not 16-byte aligned";
    default: return "unknown status";
    }
}

int tasq_stage_of_step(int t, int S, int T)
{
    if (S < 1 || T < 1 || S > T || t < 0 || t >= T)
        return TASQ_ERR_RANGE;
    return (int)(((long long)t * S) / T);
}

size_t tasq_planes_bytes(int N, int K)
{
    return (size_t)tasq::planes_bytes_host(N, K);
}

size_t tasq_workspace_bytes(int M, int N, int K)
{
    if (M <= 0 || N <= 0 || K <= 128)
        return 0;
    const int s = auto_splits(M, N, K);
    if (s < 2)
        return 0;
    int kchunk, splits;
    split_geometry(K, s, kchunk, splits);
    const unsigned long long need = 4ULL * splits * (unsigned long long)M * N;
    return need < (1ULL << 31) ? (size_t)need : 0;
}

int tasq_masked_linear(const int8_t *X, const int8_t *W, float sx, const float *sw,
                       const float *bias, int M, int N, int K, int b, int32_t *acc_out,
                       float *y_out, const tasq_opts *opts, void *stream)
{
    tasq_layer L;
    std::memset(&L, 0, sizeof L);
    L.kind = TASQ_KIND_LINEAR;
    L.M = M;
    L.N = N;
    L.K = K;
    L.sx = sx;
    L.X = X;
    L.W = W;
    L.sw = sw;
    L.bias = bias;
    L.acc = acc_out;
    L.y = y_out;
    if (int rc = check_tuning(opts))
        return rc;
    if (int rc = validate_layer(L, opts))
        return rc;
    if (b < 1 || b > 8)
        return TASQ_ERR_BITS;
    LayerDesc d = make_desc(L, opts);
    d.bits = b;
    return launch_layer(d, opts, static_cast<hipStream_t>(stream), true);
}

int tasq_masked_conv3x3(const int8_t *X, const int8_t *W, float sx, const float *sw,
                        const float *bias, int H, int Wd, int C, int N, int b,
                        int32_t *acc_out, float *y_out, const tasq_opts *opts, void *stream)
{
    if (H < 0 || Wd < 0 || C < 0 || N < 0)
        return TASQ_ERR_DIM;
    const long long M = (long long)H * Wd, K = 9LL * C;
    if (M > 0x7fffffffLL)
        return TASQ_ERR_DIM;
    if (K > TASQ_MAX_K)
        return TASQ_ERR_OVERFLOW;
    tasq_layer L;
    std::memset(&L, 0, sizeof L);
    L.kind = TASQ_KIND_CONV3X3;
    L.M = (int)M;
    L.N = N;
    L.K = (int)K;
    L.H = H;
    L.Wd = Wd;
    L.C = C;
    L.sx = sx;
    L.X = X;
    L.W = W;
    L.sw = sw;
    L.bias = bias;
    L.acc = acc_out;
    L.y = y_out;
    if (int rc = check_tuning(opts))
        return rc;
    if (int rc = validate_layer(L, opts))
        return rc;
    if (b < 1 || b > 8)
        return TASQ_ERR_BITS;
    LayerDesc d = make_desc(L, opts);
    d.bits = b;
    return launch_layer(d, opts, static_cast<hipStream_t>(stream), true);
}

int tasq_pack_planes(const int8_t *W, int N, int K, uint32_t *planes_out, void *stream)
{
    if (!W || !planes_out)
        return TASQ_ERR_NULL;
    if (N < 0 || K < 0)
        return TASQ_ERR_DIM;
    if (N == 0 || K == 0)
        return TASQ_OK;
    hipError_t e = tasq::launch_pack_planes(W, N, K, planes_out, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? TASQ_OK : TASQ_ERR_HIP;
}

int tasq_pack_weights(const int8_t *W, int N, int K, int8_t *packed_out, void *stream)
{
    if (N < 0 || K < 0)
        return TASQ_ERR_DIM;
    if (K > TASQ_MAX_K)
        return TASQ_ERR_OVERFLOW;
    if (N == 0 || K == 0)
        return TASQ_OK;
    if (!W || !packed_out)
        return TASQ_ERR_NULL;
    if (!aligned16(packed_out))
        return TASQ_ERR_ALIGN;
    hipError_t e = tasq::launch_pack_weights(W, N, K, packed_out, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? TASQ_OK : TASQ_ERR_HIP;
}

int tasq_quantize_activations(const float *x, int M, int K, int8_t *X_out, float *act_params,
                              void *stream)
{
    if (M < 0 || K < 0)
        return TASQ_ERR_DIM;
    const long long n = (long long)M * K;
    if (n == 0)
        return TASQ_OK;
    if (!x || !X_out || !act_params)
        return TASQ_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(x) & 3) || (reinterpret_cast<uintptr_t>(act_params) & 3))
        return TASQ_ERR_ALIGN;
    hipError_t e = tasq::launch_quantize_activations(x, n, X_out, act_params,
                                                     static_cast<hipStream_t>(stream));
    return e == hipSuccess ? TASQ_OK : TASQ_ERR_HIP;
}

int tasq_quantize_activations_batch(const tasq_act_job *jobs, int n, void *stream)
{
    if (n < 0)
        return TASQ_ERR_RANGE;
    if (n == 0)
        return TASQ_OK;
    if (!jobs)
        return TASQ_ERR_NULL;
    std::vector<tasq::ActJob> js;
    std::vector<const float *> bufs;
    js.reserve((size_t)n);
    bufs.reserve((size_t)n);
    for (int j = 0; j < n; ++j) {
        const tasq_act_job &a = jobs[j];
        if (a.M < 0 || a.K < 0)
            return TASQ_ERR_DIM;
        if ((long long)a.M * a.K == 0)
            continue;
        if (!a.x || !a.X_out || !a.act_params)
            return TASQ_ERR_NULL;
        if ((reinterpret_cast<uintptr_t>(a.x) & 3) || (reinterpret_cast<uintptr_t>(a.act_params) & 3))
            return TASQ_ERR_ALIGN;
        js.push_back({a.x, a.M, a.K, a.X_out, a.act_params});
        bufs.push_back(a.act_params);
    }
    std::sort(bufs.begin(), bufs.end());
    if (std::adjacent_find(bufs.begin(), bufs.end()) != bufs.end())
        return TASQ_ERR_RANGE;
    hipError_t e = tasq::launch_quantize_activations_batch(js.data(), (int)js.size(),
                                                           static_cast<hipStream_t>(stream));
    return e == hipSuccess ? TASQ_OK : TASQ_ERR_HIP;
}

int tasq_quantize_weights(const float *W, int N, int K, int8_t *W_out, float *alpha_out,
                          float *z_out, float *sw_out, void *stream)
{
    if (N < 0 || K < 0 || (N > 0 && K == 0))
        return TASQ_ERR_DIM;
    if (K > TASQ_MAX_K)
        return TASQ_ERR_OVERFLOW;
    if (N == 0)
        return TASQ_OK;
    if (!W || !W_out || !alpha_out || !z_out || !sw_out)
        return TASQ_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(W) & 3) || (reinterpret_cast<uintptr_t>(alpha_out) & 3) ||
        (reinterpret_cast<uintptr_t>(z_out) & 3) || (reinterpret_cast<uintptr_t>(sw_out) & 3))
        return TASQ_ERR_ALIGN;
    hipError_t e = tasq::launch_quantize_weights(W, N, K, W_out, alpha_out, z_out, sw_out,
                                                 static_cast<hipStream_t>(stream));
    return e == hipSuccess ? TASQ_OK : TASQ_ERR_HIP;
}

int tasq_row_sums(const int8_t *X, int M, int K, int32_t *out, void *stream)
{
    if (M < 0 || K < 0)
        return TASQ_ERR_DIM;
    if (K > TASQ_MAX_K)
        return TASQ_ERR_OVERFLOW;
    if (M == 0)
        return TASQ_OK;
    if (!out || (K > 0 && !X))
        return TASQ_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(out) & 3)
        return TASQ_ERR_ALIGN;
    hipError_t e = tasq::launch_row_sums(X, M, K, out, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? TASQ_OK : TASQ_ERR_HIP;
}

static int check_lowrank_down(const float *x, int M, int K, const uint16_t *down, int r,
                              const float *T_out)
{
    if (M < 0 || K < 0 || (r != 16 && r != 32))
        return TASQ_ERR_DIM;
    if ((long long)M * r * 4 >= (1LL << 31) || K > (1 << 30) / 32)
        return TASQ_ERR_DIM;
    if (M == 0)
        return TASQ_OK;
    if (!T_out || (K > 0 && (!x || !down)))
        return TASQ_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(x) & 3) || (reinterpret_cast<uintptr_t>(down) & 1) ||
        (reinterpret_cast<uintptr_t>(T_out) & 3))
        return TASQ_ERR_ALIGN;
    return TASQ_OK;
}

int tasq_lowrank_down(const float *x, int M, int K, const uint16_t *down, int r, float *T_out,
                      void *stream)
{
    if (int rc = check_lowrank_down(x, M, K, down, r, T_out))
        return rc;
    if (M == 0)
        return TASQ_OK;
    hipError_t e = tasq::launch_lowrank_down(x, M, K, down, r, T_out, nullptr, nullptr,
                                             static_cast<hipStream_t>(stream));
    return e == hipSuccess ? TASQ_OK : TASQ_ERR_HIP;
}

int tasq_quantize_activations_lowrank(const float *x, int M, int K, int8_t *X_out,
                                      float *act_params, const uint16_t *down, int r,
                                      float *T_out, void *stream)
{
    if (int rc = check_lowrank_down(x, M, K, down, r, T_out))
        return rc;
    if (M == 0)
        return TASQ_OK;
    if (K == 0) {       // no codes to write; the projection is zero
        hipError_t e = tasq::launch_lowrank_down(x, M, K, down, r, T_out, nullptr, nullptr,
                                                 static_cast<hipStream_t>(stream));
        return e == hipSuccess ? TASQ_OK : TASQ_ERR_HIP;
    }
    if (!X_out || !act_params)
        return TASQ_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(act_params) & 3)
        return TASQ_ERR_ALIGN;
    hipError_t e = tasq::launch_quantize_activations_lowrank(
        x, M, K, X_out, act_params, down, r, T_out, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? TASQ_OK : TASQ_ERR_HIP;
}

int tasq_weight_colsums(const int8_t *W, int N, int K, int32_t *colsums_out, void *stream)
{
    if (N < 0 || K < 0)
        return TASQ_ERR_DIM;
    if (K > TASQ_MAX_K)
        return TASQ_ERR_OVERFLOW;
    if (N == 0)
        return TASQ_OK;
    if (!colsums_out || (K > 0 && !W))
        return TASQ_ERR_NULL;
    hipError_t e = tasq::launch_weight_colsums(W, N, K, colsums_out,
                                               static_cast<hipStream_t>(stream));
    return e == hipSuccess ? TASQ_OK : TASQ_ERR_HIP;
}

size_t tasq_packed_weight_bytes(int N, int K)
{
    return (size_t)tasq::packed_weight_bytes_host(N, K);
}

size_t tasq_schedule_workspace_bytes(const tasq_layer *layers, int L)
{
    if (L <= 0)
        return 0;
    return schedule_partials_offset(L) + (layers ? round_up(max_split_bytes(layers, L), kWsAlign)
                                                 : 0);
}

// step_events[i] (caller-created hipEvent_t), when the caller asked for them.
static int record_step_event(const tasq_opts *o, int i, hipStream_t st)
{
    if (!o || !o->step_events)
        return TASQ_OK;
    return hipEventRecord(static_cast<hipEvent_t>(o->step_events[i]), st) == hipSuccess
               ? TASQ_OK
               : TASQ_ERR_HIP;
}

// static_ws: the per-device scratch array (tasq_run_schedule_noalloc) in
// place of the caller's workspace; it holds the layer list and the table
// only, so layers that a workspace schedule would split-K run unsplit.
static int run_schedule_impl(const tasq_layer *layers, int L, const uint8_t *b_table, int S,
                             int T, int t_begin, int t_end, const tasq_opts *opts, void *stream,
                             bool use_static)
{
    if (L < 0)
        return TASQ_ERR_RANGE;
    if (L > 0 && (!layers || !b_table))
        return TASQ_ERR_NULL;
    if (S < 1 || T < 1 || S > T || t_begin < 0 || t_begin > t_end || t_end > T)
        return TASQ_ERR_RANGE;
    if (S > 64)
        return TASQ_ERR_RANGE;
    if (opts && opts->workspace && (reinterpret_cast<uintptr_t>(opts->workspace) % kWsAlign))
        return TASQ_ERR_ALIGN;
    if (int rc = check_tuning(opts))
        return rc;
    for (int l = 0; l < L; ++l) {
        if (int rc = validate_layer(layers[l], opts))
            return rc;
        for (int s = 0; s < S; ++s) {
            const int b = b_table[(size_t)l * S + s];
            if (b < 1 || b > 8)
                return TASQ_ERR_BITS;
        }
    }
    if (use_static && L > TASQ_STATIC_MAX_LAYERS)
        return TASQ_ERR_WORKSPACE;
    if (L == 0 || t_begin == t_end)
        return TASQ_OK;
    hipStream_t st = static_cast<hipStream_t>(stream);
    void *static_ws = nullptr;
    if (use_static) {
        if (int rc = static_scratch(st, &static_ws))
            return rc;
    }

    std::vector<LayerDesc> descs(L);
    for (int l = 0; l < L; ++l)
        descs[l] = make_desc(layers[l], opts);

    // Grouped path: one launch per step over every layer's tiles, with the
    // layer list and bit table resident in the caller's workspace.
    // Grouped launches need the workspace for the device-side layer list.
    // Three kinds, each over every layer's work units in one launch per step:
    //  - weight streaming, when every layer is skinny (M <= 64) with the same
    //    weight source: one unit per 32 output channels;
    //  - packed-weight GEMM, when every layer has a packed weight;
    //  - staged GEMM, when every layer has its aligned row-major weight.
    // Otherwise each layer is launched on its own.
    const size_t need = use_static ? schedule_partials_offset(L)
                                   : tasq_schedule_workspace_bytes(layers, L);
    char *const ws = use_static ? static_cast<char *>(static_ws)
                                : static_cast<char *>(opts ? opts->workspace : nullptr);
    const size_t ws_bytes = use_static ? kStaticScratchBytes : (opts ? opts->workspace_bytes : 0);
    const bool have_ws = ws && ws_bytes >= need;
    // The weight copy each layer reads (AUTO: by shape, see weight_source),
    // with "some b below 8" taken over the stages the steps touch.
    const int s_first = tasq_stage_of_step(t_begin, S, T);
    const int s_last = tasq_stage_of_step(t_end - 1, S, T);
    std::vector<WeightSrc> wsrc(L);
    for (int l = 0; l < L; ++l) {
        bool below8 = false;
        for (int s = s_first; s <= s_last; ++s)
            below8 = below8 || b_table[(size_t)l * S + s] < 8;
        wsrc[l] = weight_source(descs[l], opts, below8, true);
    }
    // Only layers with a product to compute (M, N and K all positive) take
    // part in a grouped launch and decide its form; a layer with outputs
    // but K = 0 writes its bias (or zero) through the single-layer launcher
    // each step, and a layer without outputs has nothing to do.
    auto multiplies = [](const LayerDesc &d) { return d.M > 0 && d.N > 0 && d.K > 0; };
    tasq::SkinnyWeights src = tasq::SKINNY_ROWS;
    bool all_skinny = have_ws;
    bool seen = false;
    int max_m = 0;
    for (int l = 0; all_skinny && l < L; ++l) {
        if (!multiplies(descs[l]))
            continue;
        tasq::SkinnyWeights sl;
        all_skinny = skinny_source(descs[l], wsrc[l], sl) && (!seen || sl == src);
        src = sl;
        seen = true;
        max_m = descs[l].M > max_m ? descs[l].M : max_m;
    }
    bool all_packed = true;
    for (int l = 0; l < L; ++l)
        all_packed = all_packed && (!multiplies(descs[l]) ||
                                    (wsrc[l] == SRC_PACKED && packed_fits(descs[l])));
    const int v = variant_of_opts(opts);
    bool grouped = have_ws && v != TASQ_VARIANT_BITPLANE;
    for (int l = 0; grouped && l < L; ++l) {
        const LayerDesc &d = descs[l];
        if (!multiplies(d))
            continue;
        const bool staged = v != TASQ_VARIANT_PACKED && wsrc[l] != SRC_PLANES && d.W &&
                            aligned16(d.W);
        grouped = x_aligned(d) && (all_packed || staged);
    }
    if (all_skinny || grouped) {
        for (int l = 0; l < L; ++l)
            descs[l].layer = l;
        // A layer whose one 256x256 tile costs more than a compute unit's
        // even share of the step, and that split-K can cut (a long K on few
        // tiles: the 3x3 conv of the UNet block), is launched on its own
        // each step, split-K over the partials room of the workspace, ahead
        // of the grouped launch over the other layers; inside the grouped
        // launch its tiles would set the step time and force small tiles on
        // every layer (SDXL-Turbo-shaped block: 174.5 us per step grouped,
        // 99.1 + 39.1 us split this way).
        std::vector<LayerDesc> solo;
        {
            std::vector<LayerDesc> rest;
            for (const LayerDesc &d : descs) {
                if (multiplies(d))
                    rest.push_back(d);
                else if (d.M > 0 && d.N > 0)
                    solo.push_back(d);
            }
            descs.swap(rest);
        }
        if (!all_skinny && !all_packed) {
            double ops = 0;
            for (const LayerDesc &d : descs)
                ops += 2.0 * d.M * (double)d.N * d.K;
            std::vector<LayerDesc> rest, split;
            for (const LayerDesc &d : descs) {
                const bool long_tile = 2.0 * 256 * 256 * (double)d.K > ops / kComputeUnits;
                if (long_tile && auto_splits(d.M, d.N, d.K) > 1)
                    split.push_back(d);
                else
                    rest.push_back(d);
            }
            if (!rest.empty() && !split.empty()) {
                descs.swap(rest);
                solo.insert(solo.end(), split.begin(), split.end());
            }
        }
        // Weight streaming: the workgroups of the deepest layers first.  A
        // workgroup streams all of its layer's K, so the 4608-deep layers'
        // workgroups run four times as long as the 1152-deep ones; launched
        // last (in layer order) they leave the end of the step to a few
        // compute units (28-block PixArt-shaped step at 16 tokens, planes:
        // 0.0581 ms ordered by K, 0.0638 ms in layer order).
        if (all_skinny)
            std::stable_sort(descs.begin(), descs.end(),
                             [](const LayerDesc &x, const LayerDesc &y) { return x.K > y.K; });
        const int LG = (int)descs.size();
        bool any_conv = false;
        for (int l = 0; l < LG; ++l)
            any_conv = any_conv || descs[l].kind == tasq::KIND_CONV3X3;
        tasq::TileShape ts = {32, 32, 128};
        hipError_t (*launch_step)(const LayerDesc *, int, int, const uint8_t *, int, int, bool,
                                  hipStream_t) = nullptr;
        hipError_t (*launch_persistent)(const LayerDesc *, int, int, const tasq::XcdRuns &,
                                        const uint8_t *, int, int, int, int,
                                        hipStream_t) = nullptr;
        bool big_tile = false;      // the 256x256 tile, which AUTO runs persistent
        bool extras = false;
        for (int l = 0; l < LG; ++l)
            extras = extras || descs[l].lr_T != nullptr || descs[l].wz != nullptr;
        if (all_skinny) {
            // one unit per 32 output channels, all tokens
            ts = {tasq::kSkinnyMaxM, 32, 128};
        } else if (all_packed) {
            const int ptile = pick_packed_grouped_tile(opts);
            const tasq::PackedTileOps &ops = tasq::packed_tile_ops(ptile);
            ts = ops.shape;
            launch_step = ops.grouped;
            if (!any_conv && !extras)
                launch_persistent = ops.persistent;
            big_tile = ptile == tasq::PTILE_256x256_K128_W8;
        } else {
            const int tile = pick_grouped_tile(opts, descs);
            const tasq::TileOps &ops = tasq::tile_ops(tile);
            ts = ops.shape;
            launch_step = ops.grouped;
            if (!any_conv)
                launch_persistent = extras ? ops.persistent_extras : ops.persistent;
            big_tile = tile == tasq::TILE_256x256_K128_W8_PF1;
        }
        long long total = 0;
        for (int l = 0; l < LG; ++l) {
            LayerDesc &d = descs[l];
            d.tiles_m = (d.M + ts.bm - 1) / ts.bm;
            d.tiles_n = (d.N + ts.bn - 1) / ts.bn;
            d.tile_first = 0;
            d.tile_begin = (int)total;
            total += (long long)d.tiles_m * d.tiles_n;
            if (total > 0x7fffffffLL)
                return TASQ_ERR_DIM;
        }
        if (total == 0 && solo.empty())
            return TASQ_OK;
        if (!use_persistent(opts, big_tile, total))
            launch_persistent = nullptr;
        const int wgs_per_xcd = persistent_wgs_per_xcd(opts);
        const int parties = persistent_parties(opts, wgs_per_xcd);
        // The GEMM kernels give each XCD one contiguous run of the work
        // units (for L2 locality): the persistent launch runs of about equal
        // cost (cost_runs), the one-workgroup-per-tile launches runs equal in
        // count.  For the latter, when the layers' tiles differ in cost (K)
        // and the layer order leaves one run much heavier than the others,
        // every layer is cut into kXcds rounds instead, so that each run
        // holds about an eighth of every layer (measured slower than
        // contiguous runs for the persistent step: 4.27 against 4.15 ms).
        std::vector<LayerDesc> segs;
        if (!all_skinny && !launch_persistent &&
            xcd_imbalance(descs, total) > kImbalanceLimit) {
            segs.reserve((size_t)LG * kXcds);
            long long begin = 0;
            for (int r = 0; r < kXcds; ++r)
                for (int l = 0; l < LG; ++l) {
                    const long long n = (long long)descs[l].tiles_m * descs[l].tiles_n;
                    const long long lo = n * r / kXcds, hi = n * (r + 1) / kXcds;
                    if (hi <= lo)
                        continue;
                    LayerDesc d = descs[l];
                    d.tile_first = (int)lo;
                    d.tile_begin = (int)begin;
                    begin += hi - lo;
                    segs.push_back(d);
                }
        } else {
            segs = descs;
        }
        const int nseg = (int)segs.size();
        const tasq::XcdRuns runs = cost_runs(segs, total);
        LayerDesc *d_descs = reinterpret_cast<LayerDesc *>(ws);
        uint8_t *d_table = reinterpret_cast<uint8_t *>(
            ws + round_up((size_t)L * kXcds * sizeof(LayerDesc), kWsAlign));
        std::vector<uint8_t> table((size_t)L * 64, 0);
        for (int l = 0; l < L; ++l)
            for (int s = 0; s < S; ++s)
                table[(size_t)l * S + s] = b_table[(size_t)l * S + s];
        if (hipMemcpyAsync(d_descs, segs.data(), (size_t)nseg * sizeof(LayerDesc),
                           hipMemcpyHostToDevice, st) != hipSuccess)
            return TASQ_ERR_HIP;
        if (hipMemcpyAsync(d_table, table.data(), (size_t)L * S, hipMemcpyHostToDevice, st) !=
            hipSuccess)
            return TASQ_ERR_HIP;
        // Schedules ignore split_k: a layer launched on its own takes the
        // automatic split over the partials room, which
        // tasq_schedule_workspace_bytes reserved for it.
        tasq_opts sopts = opts ? *opts : tasq_opts{};
        sopts.split_k = 0;
        sopts.step_events = nullptr;
        sopts.workspace = use_static ? nullptr : ws + schedule_partials_offset(L);
        sopts.workspace_bytes = use_static ? 0 : ws_bytes - schedule_partials_offset(L);
        for (int t = t_begin; t < t_end; ++t) {
            const int s = tasq_stage_of_step(t, S, T);
            if (int rc = record_step_event(opts, 2 * (t - t_begin), st))
                return rc;
            for (LayerDesc d : solo) {
                d.bits = b_table[(size_t)d.layer * S + s];
                if (int rc = launch_layer(d, &sopts, st, true))
                    return rc;
            }
            if (total == 0) {
                if (int rc = record_step_event(opts, 2 * (t - t_begin) + 1, st))
                    return rc;
                continue;
            }
            const hipError_t e =
                all_skinny ? tasq::launch_skinny_grouped(d_descs, nseg, (int)total, max_m, src,
                                                         d_table, S, s, st)
                : launch_persistent
                    ? launch_persistent(d_descs, nseg, (int)total, runs, d_table, S, s,
                                        wgs_per_xcd, parties, st)
                    : launch_step(d_descs, nseg, (int)total, d_table, S, s, any_conv, st);
            if (e != hipSuccess)
                return TASQ_ERR_HIP;
            if (int rc = record_step_event(opts, 2 * (t - t_begin) + 1, st))
                return rc;
        }
        return TASQ_OK;
    }

    for (int t = t_begin; t < t_end; ++t) {
        const int s = tasq_stage_of_step(t, S, T);
        if (int rc = record_step_event(opts, 2 * (t - t_begin), st))
            return rc;
        for (int l = 0; l < L; ++l) {
            descs[l].bits = b_table[(size_t)l * S + s];
            if (int rc = launch_layer(descs[l], opts, st))
                return rc;
        }
        if (int rc = record_step_event(opts, 2 * (t - t_begin) + 1, st))
            return rc;
    }
    return TASQ_OK;
}

// The host-side lists (layer descriptors, segments, the table copy) are
// std::vectors: running out of host memory is returned as TASQ_ERR_HIP, not
// thrown across the C ABI.
int tasq_run_schedule(const tasq_layer *layers, int L, const uint8_t *b_table, int S, int T,
                      int t_begin, int t_end, const tasq_opts *opts, void *stream)
{
    try {
        return run_schedule_impl(layers, L, b_table, S, T, t_begin, t_end, opts, stream, false);
    } catch (const std::bad_alloc &) {
        return TASQ_ERR_HIP;
    }
}

int tasq_run_schedule_noalloc(const tasq_layer *layers, int L, const uint8_t *b_table, int S,
                              int T, int t_begin, int t_end, const tasq_opts *opts, void *stream)
{
    try {
        return run_schedule_impl(layers, L, b_table, S, T, t_begin, t_end, opts, stream, true);
    } catch (const std::bad_alloc &) {
        return TASQ_ERR_HIP;
    }
}

}  // extern "C"
