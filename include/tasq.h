/*
 * tasq.h - C ABI of the TASQ masked quantized linear layer for MI355X (gfx950).
 *
 * The operation (TASQ, arxiv 2608.03057):
 *   - one stored 8-bit weight buffer W per layer, shared by every denoising
 *     stage (Sec. 3.2; Sec. 4.3 "Deployment procedure");
 *   - at stage s, layer l runs at effective precision b = table[l][s]
 *     (Sec. 1 and App. G.1: switching precision is a table lookup, the kernel
 *     takes the number of bit planes as an argument);
 *   - the operand is the stored code with its k = 8 - b least significant
 *     bits removed and the scale kept: W_b = 2^k * floor(W / 2^k)
 *     (Sec. 3.1 Eq. truncquant, Sec. 3.2.1 Eq. lsb_masking, App. G.2
 *     Eqs. hw_rightshift and hw_multi_lsb);
 *   - acc = X * W_b^T accumulated exactly in int32 (Sec. 3.1 Eq. qalora with
 *     the LoRA branch merged), then y = acc * sx * sw[n] (+ bias[n]) in fp32
 *     (App. A.1 dequantisation, zero points zero, the 2^n/(2^n-1) weight
 *     factor folded into sw).
 *
 * Conventions for every entry point:
 *   - Tensor pointers are DEVICE memory owned by the caller.  The library
 *     never frees, retains past the call, or writes its inputs.  Host
 *     pointers (the layer array, the bit table) are read during the call
 *     only.
 *   - Layouts are row-major: X int8 [M][K], W int8 [N][K] (output x input,
 *     K contiguous), acc int32 [M][N], y fp32 [M][N]; sw, bias fp32 [N].
 *   - `stream` is a hipStream_t (NULL = the default stream).  Calls are
 *     asynchronous and stream-ordered; results are visible after the stream
 *     is synchronised.  Device faults surface at that synchronisation.
 *   - Every argument (for a schedule: every layer and every table entry) is
 *     validated before any work is enqueued; on an error return nothing was
 *     enqueued and outputs are untouched.  No C++ exception crosses the ABI.
 *   - Calls on different streams that share output buffers race; calls that
 *     share a workspace must be ordered on one stream.
 */
#ifndef TASQ_H
#define TASQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes: 0 on success, negative on error. */
enum {
    TASQ_OK = 0,
    TASQ_ERR_NULL = -1,      /* a required pointer is NULL, or no output requested */
    TASQ_ERR_DIM = -2,       /* a dimension is negative or inconsistent           */
    TASQ_ERR_BITS = -3,      /* b (or a table entry) outside [1, 8]                */
    TASQ_ERR_OVERFLOW = -4,  /* K > TASQ_MAX_K: int32 accumulation could overflow  */
    TASQ_ERR_RANGE = -5,     /* bad S, T, t_begin, t_end, L or job count, or an
                                act_params shared by two jobs of a batch          */
    TASQ_ERR_LAYOUT = -6,    /* requested variant needs a layout that is absent    */
    TASQ_ERR_WORKSPACE = -7, /* workspace missing or smaller than required         */
    TASQ_ERR_HIP = -8,       /* a HIP call or launch failed, or host memory ran out */
    TASQ_ERR_KIND = -9,      /* unknown layer kind or variant                       */
    TASQ_ERR_ALIGN = -10     /* workspace not 256-byte aligned, or a packed weight
                                not 16-byte aligned                                */
};

/* |X| <= 128 and |W_b| <= 128, so |acc| <= 16384 * K < 2^31 iff K <= 131071. */
#define TASQ_MAX_K 131071

/* Length in floats of the parameter buffer of an asymmetric activation
 * tensor (tasq_quantize_activations): [0] alpha, [1] z, the rest scratch. */
#define TASQ_ACT_PARAMS_FLOATS 1028

/* Kernel variants (tasq_opts.variant). */
enum {
    TASQ_VARIANT_AUTO = 0,      /* library picks per shape                         */
    TASQ_VARIANT_MASKED_I8 = 1, /* int8 MFMA GEMM, mask fused into weight staging  */
    TASQ_VARIANT_BITPLANE = 2,  /* reads only the top b planes of W_planes         */
    TASQ_VARIANT_PACKED = 3     /* int8 MFMA GEMM on W_packed (tasq_pack_weights)  */
};

/* Layer kinds (tasq_layer.kind). */
enum {
    TASQ_KIND_LINEAR = 0,       /* X [M][K]                                        */
    TASQ_KIND_CONV3X3 = 1       /* X NHWC [H][Wd][C], W [N][3][3][C], stride 1,
                                   zero padding 1; M = H*Wd, K = 9*C               */
};

/*
 * Optional controls; pass NULL for defaults (AUTO variant, no workspace).
 *   variant         TASQ_VARIANT_*.
 *   split_k         single-layer calls with the row-major weight (not the
 *                   packed, bit-plane or weight-streaming paths): 0 = the
 *                   library may cut K into ranges when few output tiles
 *                   would leave compute units idle, and does so only when
 *                   workspace holds tasq_workspace_bytes(M, N, K) bytes;
 *                   1 = never; s >= 2 = cut K into (at most) s ranges,
 *                   which needs s*M*N*4 bytes of workspace
 *                   (TASQ_ERR_WORKSPACE otherwise).  The ranges' int32
 *                   partial sums are added in a fixed order, so every
 *                   output is identical to the unsplit one.  Negative:
 *                   TASQ_ERR_RANGE.  Schedules ignore it (a long-K layer
 *                   that a schedule launches on its own uses the automatic
 *                   split over the schedule workspace).
 *   W_planes        bit-plane copy of W as written by tasq_pack_planes; needed
 *                   by the BITPLANE variant (W may then be NULL).
 *   W_packed        W in the MFMA operand order as written by
 *                   tasq_pack_weights; used by the PACKED variant and chosen
 *                   by AUTO when present (W may then be NULL).
 *   workspace       device scratch, 256-byte aligned, owned by the caller;
 *                   holds the schedule's device-side layer list and bit
 *                   table (size from tasq_schedule_workspace_bytes), or a
 *                   single layer's split-K partial sums (split_k).
 *                   Contents need no initialisation and are left
 *                   unspecified.
 *   workspace_bytes its size in bytes.
 *   act_params      device float[TASQ_ACT_PARAMS_FLOATS] written by
 *                   tasq_quantize_activations, or NULL.  When given, X holds
 *                   asymmetric activation codes (stored as Q - 128), sx is
 *                   ignored, and (only [0] and [1] are read)
 *                   y = act_params[0] * sw[n] *
 *                       (acc + (128 - act_params[1]) * colsums[b-1][n]) + bias[n]
 *                   (App. A.1.2 dequantisation x_hat = alpha (Q - z)).
 *   colsums         device int32 [8][N] from tasq_weight_colsums; required
 *                   with act_params.  act_params and colsums must be 4-byte
 *                   aligned (TASQ_ERR_ALIGN).  Linear layers only: a conv's
 *                   zero padding is not the code of a real zero, so
 *                   act_params on a TASQ_KIND_CONV3X3 layer or in
 *                   tasq_masked_conv3x3 is TASQ_ERR_LAYOUT.
 *   lowrank_T       device fp32 [M][lowrank_rank] from tasq_lowrank_down (or
 *                   tasq_quantize_activations_lowrank), or NULL: the 16-bit
 *                   low-rank branch of an SVDQuant-initialised layer (Sec.
 *                   4.1 setup, training-details appendix).  When given, y
 *                   gains (lowrank_T lowrank_up^T)[m][n]; acc is unchanged.
 *   lowrank_up      device bfloat16 [N][lowrank_rank], the branch's up
 *                   projection (bit patterns); required with lowrank_T.
 *   lowrank_rank    16 or 32 (TASQ_ERR_DIM otherwise).  lowrank_T and
 *                   lowrank_up must be 16-byte aligned (TASQ_ERR_ALIGN);
 *                   linear layers only (TASQ_ERR_LAYOUT on a conv).
 *   w_zero          device fp32 [N] per-channel weight zero points from
 *                   tasq_quantize_weights, or NULL (zero points 0).  When
 *                   given, W holds the codes Q - 128 of App. A.1.1, sw the
 *                   factor 256/255 alpha, and the masked weight dequantises
 *                   to sw[n] (W_b + 128 - w_zero[n]), so y gains
 *                   scale * (128 - w_zero[n]) * R[m] inside the dequantised
 *                   sum, R[m] = x_rowsums[m] (+ K (128 - z) with
 *                   act_params).  acc is unchanged.
 *   x_rowsums       device int32 [M] from tasq_row_sums of X; required with
 *                   w_zero.  Both 4-byte aligned (TASQ_ERR_ALIGN); linear
 *                   layers only (TASQ_ERR_LAYOUT on a conv).
 * Tuning overrides, for sweeps and tests (0 everywhere = the library's own
 * choice, which every other caller should keep):
 *   tile            t + 1 forces staged-weight tile TASQ_TILE_* t (single
 *                   calls, split-K and grouped schedule steps).
 *   packed_tile     t + 1 forces packed-weight tile TASQ_PTILE_* t.
 *   persistent      grouped schedule steps over linear layers (with
 *                   low-rank or weight-zero-point terms only on row-major
 *                   weights and the TASQ_TILE_256x256_K128_W8 tile): 1 = one
 *                   workgroup per output tile, 2 = the persistent launch
 *                   (one workgroup per compute unit walking a run of tiles),
 *                   whatever the tile and the tile count.
 *   persistent_wgs  workgroups per XCD of the persistent launch (1..1024;
 *                   0 = one per compute unit, 32).
 *   persistent_parties  parts of each XCD's run of tiles walked side by side
 *                   by the persistent launch (it must divide the workgroups
 *                   per XCD, else 1 is used; 0 = 1).
 *   Out of range: TASQ_ERR_RANGE.
 * Measurement:
 *   step_events     tasq_run_schedule only: NULL, or a host array of
 *                   2 * (t_end - t_begin) hipEvent_t created by the caller;
 *                   the library records step_events[2i] on the stream right
 *                   before the kernels of step t_begin + i and
 *                   step_events[2i + 1] right after them, so the pair times
 *                   that step's launches alone (not the per-call upload of
 *                   the layer list).  A failed record is TASQ_ERR_HIP.
 */

/* Staged-weight tile configurations (tasq_opts.tile - 1): output tile,
 * K bytes per step, waves per workgroup. */
enum {
    TASQ_TILE_256x256_K128_W8 = 0,
    TASQ_TILE_256x256_K64_W8 = 1,
    TASQ_TILE_128x128_K128_W4 = 2,
    TASQ_TILE_64x64_K128_W4 = 3,
    TASQ_TILE_256x128_K64_W4 = 4,
    TASQ_TILE_128x256_K64_W4 = 5,
    TASQ_TILE_COUNT = 6
};

/* Packed-weight tile configurations (tasq_opts.packed_tile - 1). */
enum {
    TASQ_PTILE_256x256_K128_W8 = 0,
    TASQ_PTILE_256x256_K64_W8 = 1,
    TASQ_PTILE_128x256_K128_W4 = 2,
    TASQ_PTILE_128x256_K64_W4 = 3,
    TASQ_PTILE_256x128_K64_W4 = 4,
    TASQ_PTILE_128x128_K64_W4 = 5,
    TASQ_PTILE_64x64_K128_W4 = 6,
    TASQ_PTILE_COUNT = 7
};
typedef struct tasq_opts {
    int32_t variant;
    int32_t split_k;
    const uint32_t *W_planes;
    void *workspace;
    size_t workspace_bytes;
    const int8_t *W_packed;
    const float *act_params;
    const int32_t *colsums;
    const float *lowrank_T;
    const uint16_t *lowrank_up;
    int32_t lowrank_rank;
    const float *w_zero;
    const int32_t *x_rowsums;
    int32_t tile;
    int32_t packed_tile;
    int32_t persistent;
    int32_t persistent_wgs;
    int32_t persistent_parties;
    void **step_events;
} tasq_opts;

/*
 * y = (X * W_b^T) * sx * sw[n] (+ bias[n]),  W_b = 2^(8-b) floor(W / 2^(8-b)).
 *   X        int8 [M][K] device, activation codes (any value in [-128, 127]).
 *   W        int8 [N][K] device, stored 8-bit weight codes; may be NULL when
 *            the BITPLANE variant is requested with opts->W_planes, or when
 *            opts->W_packed is given (AUTO or PACKED variant).
 *   sx       per-tensor activation scale.
 *   sw       fp32 [N] device, per-output-channel weight scale (read only for y).
 *   bias     fp32 [N] device or NULL.
 *   M, N, K  >= 0, K <= TASQ_MAX_K; M == 0 or N == 0 enqueues nothing,
 *            K == 0 writes acc = 0 and y = bias (or 0).
 *   b        effective weight bits, 1..8 (b = 8: the stored weight itself;
 *            b = 1: the sign plane only, W_b in {-128, 0}).
 *   acc_out  int32 [M][N] device or NULL: exact accumulators.
 *   y_out    fp32 [M][N] device or NULL: dequantised output.  At least one of
 *            acc_out / y_out must be non-NULL.
 * A pointer may be NULL when its array is empty (X when M*K == 0, W when
 * N*K == 0, outputs when M*N == 0); sw is needed only with y_out.
 * Errors: TASQ_ERR_NULL, _DIM, _BITS, _OVERFLOW, _LAYOUT, _WORKSPACE, _KIND,
 * _ALIGN, _HIP.
 */
int tasq_masked_linear(const int8_t *X, const int8_t *W, float sx, const float *sw,
                       const float *bias, int M, int N, int K, int b, int32_t *acc_out,
                       float *y_out, const tasq_opts *opts, void *stream);

/*
 * The same layer applied as a 3x3 convolution, stride 1, zero padding 1,
 * batch 1, as an implicit GEMM with M = H*Wd, K = 9*C and the reduction
 * index k = (r*3 + s)*C + ci:
 *   acc[h][w][n] = sum_{r,s,ci} X[h+r-1][w+s-1][ci] * W_b[n][r][s][ci].
 *   X int8 NHWC [H][Wd][C]; W int8 [N][3][3][C]; outputs [H][Wd][N].
 * Stands in for the convolution tensors of the UNet backbone (the paper's
 * SDXL-Turbo tensor count includes them, App. D.3).
 */
int tasq_masked_conv3x3(const int8_t *X, const int8_t *W, float sx, const float *sw,
                        const float *bias, int H, int Wd, int C, int N, int b,
                        int32_t *acc_out, float *y_out, const tasq_opts *opts, void *stream);

/*
 * Bit-plane relayout of a stored weight (App. G.2: plane p holds bit p of
 * the two's-complement code, p = 0 least significant).
 *   W          int8 [N][K] device (read only).
 *   planes_out uint32 [NB][8][KB][16][4][2] device, NB = ceil(N / 32),
 *              KB = ceil(K / 128): word planes[nb][q][kb][r][w][f] is word
 *              w of channel n = 32 nb + 16 f + r in block kb of plane
 *              p = 7 - q, i.e. bits p of W[n][128*kb + e], e = 0..127.
 *              With s = e / 32, h = (e%32)/16, i = (e%16)/4, c = e%4,
 *              element e sits in word w = 2h + s/2 at bit
 *              (8c + 4(s%2) + i + p) mod 32: each word holds one
 *              16-element half of two 32-element sub-steps, and plane p's
 *              word is rotated left by p, so that the planes' bits of four
 *              consecutive elements merge with one AND-OR per plane and one
 *              rotate.  Plane q = 0 is the sign plane.  The top b planes of
 *              a 32-channel block are one contiguous run of b*KB*128 words,
 *              and words f = 0, 1 (channels n and n + 16) are adjacent.
 *              Words of channels past N and bits past K are zero.  Size
 *              tasq_planes_bytes(N, K).
 * A one-time conversion of the stored buffer, not a per-step cost.  A
 * caller that keeps only the planes (and passes W = NULL with the BITPLANE
 * variant) stores the weight once, at the same 8 bits per element.
 */
int tasq_pack_planes(const int8_t *W, int N, int K, uint32_t *planes_out, void *stream);

/* Bytes of the planes array for an N x K weight:
 * 8 * ceil(K/128) * 32 * ceil(N/32) * 16; 0 when N or K is not positive. */
size_t tasq_planes_bytes(int N, int K);

/*
 * Relayout of a stored weight into the operand order of the int8 matrix
 * instruction (the codes themselves are unchanged; the mask to b bits is
 * applied when the kernels read them, so the packed buffer is the one 8-bit
 * copy shared by every stage, Sec. 3.2 / Sec. 4.3).
 *   W           int8 [N][K] device (read only).
 *   packed_out  int8 device, tasq_packed_weight_bytes(N, K) bytes, 16-byte
 *               aligned: unit (nb, ks) of 1024 bytes, nb < ceil(N/32),
 *               ks < KS = 4 * ceil(K/128), starts at byte (nb*KS + ks)*1024;
 *               its bytes 16*l .. 16*l+15 (l = 0..63) hold
 *               W[32*nb + l%32][32*ks + 16*(l/32) .. +15].  Bytes past row N
 *               or column K are zero.
 * The kernels then fetch each 32 x 32 weight fragment with one contiguous
 * 1 KB load and need no LDS for the weights.  A one-time conversion; a
 * caller that keeps only the packed buffer (W = NULL) stores the weight once.
 * Errors: TASQ_ERR_NULL, _DIM, _OVERFLOW, _ALIGN (packed_out not 16-byte
 * aligned), _HIP.
 */
int tasq_pack_weights(const int8_t *W, int N, int K, int8_t *packed_out, void *stream);

/* Bytes of the packed weight: 32 * ceil(N/32) * 128 * ceil(K/128). */
size_t tasq_packed_weight_bytes(int N, int K);

/*
 * Asymmetric 8-bit activation quantizer, per tensor (App. A.1.2, Eqs.
 * act_quant and act_scale), the step before the masked GEMM:
 *   alpha = (max(x) - min(x)) / 255,  z = -min(x) / alpha  (z kept real),
 *   Q = clamp(round_to_nearest(x / alpha + z), 0, 255),  X_out = Q - 128.
 * The codes are decided in IEEE single precision: correctly rounded
 * division, then addition, rounding ties to even.  When max == min,
 * alpha = 1 and z = -min (every code 0, dequantising to min exactly).
 *   x           fp32 [M][K] device, finite values, 4-byte aligned (16-byte
 *               alignment, with X_out 4-byte aligned, takes vector loads).
 *   X_out       int8 [M][K] device: the signed codes Q - 128, ready as the X
 *               of tasq_masked_linear with opts->act_params.
 *   act_params  device float[TASQ_ACT_PARAMS_FLOATS]: [0] = alpha, [1] = z
 *               on completion (stream-ordered); [2..] scratch.  Nothing needs
 *               clearing beforehand; two calls that share one buffer must be
 *               ordered on one stream.
 * M*K == 0 enqueues nothing.  Errors: TASQ_ERR_NULL, _DIM, _ALIGN (x or
 * act_params not 4-byte aligned), _HIP.
 */
int tasq_quantize_activations(const float *x, int M, int K, int8_t *X_out, float *act_params,
                              void *stream);

/* One tensor of tasq_quantize_activations_batch: the arguments of one
 * tasq_quantize_activations call. */
typedef struct tasq_act_job {
    const float *x;         /* fp32 [M][K] device */
    int32_t M, K;
    int8_t *X_out;          /* int8 [M][K] device */
    float *act_params;      /* device float[TASQ_ACT_PARAMS_FLOATS] */
} tasq_act_job;

/*
 * The quantizer of tasq_quantize_activations (App. A.1.2, Eqs. act_quant
 * and act_scale) over n tensors, e.g. the inputs of every layer of one
 * denoising step, in one launch per group of up to 8 tensors (and 128 MB of
 * x) plus one, instead of 2 n launches (the range
 * pass of each group of tensors shares a launch with the code pass of the
 * group before).  Every job's codes, alpha and z equal those of a
 * tasq_quantize_activations call on it.
 *   jobs    host array of n jobs, read during the call only; each as the
 *           arguments of tasq_quantize_activations.  Jobs with M*K == 0 are
 *           skipped.  No two jobs may share an act_params buffer
 *           (TASQ_ERR_RANGE); outputs that overlap inputs or each other are
 *           the caller's error.
 *   n       number of jobs, >= 0 (TASQ_ERR_RANGE otherwise); n == 0
 *           enqueues nothing.
 * Every job is validated before anything is enqueued (TASQ_ERR_NULL, _DIM,
 * _ALIGN as for the single call).  Asynchronous on `stream`; allocates
 * nothing on the device.
 */
int tasq_quantize_activations_batch(const tasq_act_job *jobs, int n, void *stream);

/*
 * Channel sums of the masked weight at every precision, for the zero-point
 * term of asymmetric activations: colsums_out[b-1][n] = sum_k W_b[n][k],
 * b = 1..8 (int32 [8][N] device).  A one-time pass over the stored buffer,
 * like the packers.  Errors: TASQ_ERR_NULL, _DIM, _OVERFLOW, _HIP.
 */
int tasq_weight_colsums(const int8_t *W, int N, int K, int32_t *colsums_out, void *stream);

/*
 * Offline weight quantizer (App. A.1.1, Eqs. weight_quant, weight_scale,
 * weight_dequant) at the stored precision n = 8, per output channel:
 *   alpha = (max - min) / 256,  z = -min / alpha (kept real),
 *   Q = clamp(floor(w / alpha + z), 0, 255),  W_out = Q - 128,
 *   sw = alpha * 256 / 255, so that w_hat = sw * (Q - z).
 * Decided in IEEE single precision (correctly rounded division, then
 * addition, then floor); a constant row takes alpha = 1, z = -min.  The
 * 2^n grid makes every lower precision a prefix of the stored code (Eq.
 * truncquant), so W_out is the shared buffer of every stage as it is.
 *   W        fp32 [N][K] device, finite, 4-byte aligned.
 *   W_out    int8 [N][K] device: the codes, for tasq_masked_linear and the
 *            packers.
 *   alpha_out, z_out, sw_out  fp32 [N] device (z_out is the w_zero and
 *            sw_out the sw of tasq_masked_linear).
 * N == 0 enqueues nothing.  Errors: TASQ_ERR_NULL, _DIM (negative sizes,
 * K == 0 with N > 0), _OVERFLOW (K > TASQ_MAX_K), _ALIGN, _HIP.
 */
int tasq_quantize_weights(const float *W, int N, int K, int8_t *W_out, float *alpha_out,
                          float *z_out, float *sw_out, void *stream);

/* One weight of tasq_quantize_weights_batch: the arguments of one
 * tasq_quantize_weights call. */
typedef struct tasq_weight_job {
    const float *W;         /* fp32 [N][K] device */
    int32_t N, K;
    int8_t *W_out;          /* int8 [N][K] device */
    float *alpha_out, *z_out, *sw_out;  /* fp32 [N] device */
} tasq_weight_job;

/*
 * The quantizer of tasq_quantize_weights (App. A.1.1) over n weights, e.g.
 * every layer of a model, in one launch per 16 weights instead of one per
 * weight: the rows of up to 16 weights share a launch.  Every job's codes,
 * alpha, z and sw equal those of a tasq_quantize_weights call on it.
 *   jobs    host array of n jobs, read during the call only; each as the
 *           arguments of tasq_quantize_weights.  Jobs with N == 0 are
 *           skipped.  No two jobs may share an alpha_out buffer
 *           (TASQ_ERR_RANGE); other overlaps of outputs with inputs or
 *           each other are the caller's error.
 *   n       number of jobs, >= 0 (TASQ_ERR_RANGE otherwise); n == 0
 *           enqueues nothing.
 * Every job is validated before anything is enqueued (TASQ_ERR_NULL, _DIM,
 * _OVERFLOW, _ALIGN as for the single call).  Asynchronous on `stream`;
 * allocates nothing on the device.
 */
int tasq_quantize_weights_batch(const tasq_weight_job *jobs, int n, void *stream);

/*
 * Row sums of int8 activation codes, out[m] = sum_k X[m][k] (int32 [M]),
 * the x_rowsums that a weight zero point needs.  M == 0 enqueues nothing.
 * Errors: TASQ_ERR_NULL, _DIM, _OVERFLOW (K > TASQ_MAX_K), _HIP.
 */
int tasq_row_sums(const int8_t *X, int M, int K, int32_t *out, void *stream);

/*
 * Down projection of the 16-bit low-rank branch (Sec. 4.1 setup: a frozen
 * rank-16 or rank-32 branch beside the quantized weight):
 *   T[m][j] = sum_k bf16(x[m][k]) * down[j][k],
 * bf16() rounding to nearest bfloat16, ties to even; fp32 accumulation.
 *   x        fp32 [M][K] device, finite values, 4-byte aligned.
 *   down     bfloat16 [r][K] device (bit patterns), 2-byte aligned.
 *   r        16 or 32.
 *   T_out    fp32 [M][r] device, the lowrank_T of tasq_opts / tasq_layer.
 * M == 0 enqueues nothing; K == 0 writes zeros.  Errors: TASQ_ERR_NULL,
 * _DIM (negative sizes, r not 16 or 32, M*r*4 >= 2^31), _ALIGN, _HIP.
 */
int tasq_lowrank_down(const float *x, int M, int K, const uint16_t *down, int r, float *T_out,
                      void *stream);

/*
 * tasq_quantize_activations and tasq_lowrank_down of the same x in one read
 * of x: the down projection's pass also folds the range of x.  Arguments and
 * errors as in the two calls.
 */
int tasq_quantize_activations_lowrank(const float *x, int M, int K, int8_t *X_out,
                                      float *act_params, const uint16_t *down, int r,
                                      float *T_out, void *stream);

/*
 * Stage of denoising step t (Sec. 3.2: contiguous stages sharing one mask;
 * Sec. 4.1: 20 steps in four stages, or one stage per step when S = T;
 * App. D.1: stage 0 is the noisiest, first part of the trajectory):
 *   s = floor(t * S / T).
 * Returns s in [0, S), or TASQ_ERR_RANGE unless 1 <= S <= T and 0 <= t < T.
 */
int tasq_stage_of_step(int t, int S, int T);

/* One layer of a schedule.  For TASQ_KIND_LINEAR: M, N, K as in
 * tasq_masked_linear and H, Wd, C ignored.  For TASQ_KIND_CONV3X3: H, Wd, C,
 * N as in tasq_masked_conv3x3, and M, K must equal H*Wd and 9*C.
 * Pointer fields follow tasq_masked_linear. */
typedef struct tasq_layer {
    int32_t kind;
    int32_t M, N, K;
    int32_t H, Wd, C;
    float sx;
    const int8_t *X;
    const int8_t *W;
    const uint32_t *W_planes;
    const float *sw;
    const float *bias;
    int32_t *acc;
    float *y;
    const int8_t *W_packed;     /* packed copy of W or NULL (tasq_pack_weights) */
    const float *act_params;    /* asymmetric activations (see tasq_opts) or NULL */
    const int32_t *colsums;     /* [8][N] channel sums, required with act_params */
    const float *lowrank_T;     /* low-rank branch (see tasq_opts) or NULL */
    const uint16_t *lowrank_up;
    int32_t lowrank_rank;
    const float *w_zero;        /* weight zero points (see tasq_opts) or NULL */
    const int32_t *x_rowsums;
} tasq_layer;

/*
 * Runs denoising steps t = t_begin .. t_end-1 (Sec. 3.2 stage sharing;
 * App. G, per-stage precision with no re-launch or reload): for each step,
 * s = tasq_stage_of_step(t, S, T) and every layer l computes its output at
 * b = b_table[l*S + s], overwriting its acc / y buffers.  After the call the
 * buffers hold step t_end-1 (t_begin == t_end enqueues nothing).
 *   layers   host array of L layer descriptors (read during the call only).
 *   b_table  host uint8 [L][S], entries in [1, 8] (read during the call only).
 *   1 <= S <= T, 0 <= t_begin <= t_end <= T.
 * With opts->workspace of at least tasq_schedule_workspace_bytes(layers, L)
 * bytes, each step is one grouped launch over every layer's work; without it
 * each layer is launched separately.  The grouped launch streams the weights
 * (one workgroup per 32 output channels) when every layer has M <= 64 and
 * the same weight source (bit planes with the BITPLANE variant, packed
 * buffers, or row-major W); otherwise it tiles every layer's GEMM, reading
 * the packed weights when every layer carries W_packed (W may then be NULL)
 * and the row-major W otherwise.  With row-major weights, a layer whose one
 * 256x256 output tile would cost more than a compute unit's even share of
 * the step and which split-K would cut (a long K on few tiles, e.g. a 3x3
 * conv over 32x32 pixels) is launched on its own each step, split-K over the
 * partials room of the workspace, ahead of the grouped launch over the
 * other layers.  A layer with M == 0 or N == 0 does nothing, and a layer
 * with K == 0 (acc = 0, y = bias or 0, as tasq_masked_linear) is launched
 * on its own each step; neither takes part in, or decides the form of, the
 * grouped launch.  The whole table and every layer are validated before
 * anything is enqueued.
 */
int tasq_run_schedule(const tasq_layer *layers, int L, const uint8_t *b_table, int S, int T,
                      int t_begin, int t_end, const tasq_opts *opts, void *stream);

/* Limits of tasq_run_schedule_noalloc: layers per call, and the bytes of
 * the scratch array it keeps in each GPU's memory (the device layer list,
 * room for 8 segments of 176 bytes per layer, and the bit table). */
#define TASQ_STATIC_MAX_LAYERS 256
#define TASQ_STATIC_SCRATCH_BYTES 376832

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * schedule as tasq_run_schedule, with the same arguments, validation and
 * results, but the device-side layer list and bit table live in a scratch
 * array of TASQ_STATIC_SCRATCH_BYTES that the library holds in each GPU's
 * memory for the life of the process, instead of in opts->workspace (which
 * is not used).  Nothing is allocated: no hipMalloc, hipFree or allocating
 * library call; the first call on a device looks up that device's array
 * address once.
 *   L <= TASQ_STATIC_MAX_LAYERS, else TASQ_ERR_WORKSPACE (nothing enqueued).
 *   A layer that a workspace schedule would cut with split-K (a long K on
 *   few tiles) runs unsplit: same result, no partial sums to hold.
 * Every call on one GPU shares that GPU's array, and a call overwrites it
 * (stream-ordered) before its kernels read it: calls ordered on one stream
 * are safe, calls that overlap on one GPU (other streams, other host
 * threads) race on the array and must not be made.
 */
int tasq_run_schedule_noalloc(const tasq_layer *layers, int L, const uint8_t *b_table, int S,
                              int T, int t_begin, int t_end, const tasq_opts *opts,
                              void *stream);

/* Workspace with which a single layer call (split_k = 0) cuts K into ranges:
 * splits * M * N * 4 bytes, or 0 when it would not split this shape (enough
 * output tiles, or K too short).  A smaller workspace runs unsplit. */
size_t tasq_workspace_bytes(int M, int N, int K);

/* Workspace for the grouped schedule over these layers (host array): the
 * device layer list and bit table, plus the split-K partial sums of the
 * largest layer that tasq_workspace_bytes would split (0 if none). */
size_t tasq_schedule_workspace_bytes(const tasq_layer *layers, int L);

/* Static description of a status code; never NULL. */
const char *tasq_status_string(int status);

/*
 * Compute accounting of steps t_begin..t_end-1 of a schedule (same layers
 * and table as tasq_run_schedule), summed over every (layer, step) GEMM
 * with b = b_table[l][floor(t*S/T)] and MACs = M*N*K:
 *   macs                 total multiply-accumulates;
 *   b_eff                MAC-weighted mean of b, the Eff. W-bit of the
 *                        quality-compute table (Sec. 4; the paper does not
 *                        define the weighting);
 *   b_mean               plain mean of b over (layer, step);
 *   bitops               sum MACs * b * act_bits;
 *   rel_bitops           bitops / (64 macs), Rel. BitOPs against static W8A8;
 *   rel_cycles_measured  cycles relative to static 8-bit weights under the
 *                        bit-serial engine's measured law (cycles grow as
 *                        weight x activation planes, switching is free;
 *                        Tab. measured), = b_eff / 8;
 *   rel_cycles_as_a4     the same under the activation-stationary per-tile
 *                        law at 4 activation planes, 570 L + 2603 cycles
 *                        (Tab. codesign).
 * Host only; reads no device memory.  Errors: TASQ_ERR_NULL, _RANGE (S, T,
 * step range, act_bits outside 1..16), _DIM, _BITS (a table entry outside
 * 1..8).  *out is zeroed first.
 */
typedef struct tasq_cost {
    double macs;
    double b_eff;
    double b_mean;
    double bitops;
    double rel_bitops;
    double rel_cycles_measured;
    double rel_cycles_as_a4;
} tasq_cost;

int tasq_schedule_cost(const tasq_layer *layers, int L, const uint8_t *b_table, int S, int T,
                       int t_begin, int t_end, int act_bits, tasq_cost *out);

#ifdef __cplusplus
}
#endif

#endif /* TASQ_H */
