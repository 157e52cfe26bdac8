/*
 * CPU oracle for the TASQ masked quantized linear layer.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header, table or helper with
 * the HIP library.
 *
 * Every function is the plain definition written out, with no blocking,
 * fusion or reordering: integer products are accumulated in int64 in
 * ascending k, floating point is fp64.  Rows of the output are distributed
 * over OpenMP threads, which changes no arithmetic.
 *
 * Definitions followed (TASQ, arxiv 2608.03057):
 *  - truncation-consistent quantizer, Sec. 3.1 Eq. (truncquant): a lower
 *    precision code is the floor of the higher one divided by two;
 *  - k-bit generalisation, App. G.2 Eqs. (hw_rightshift, hw_multi_lsb): the
 *    b-bit operand is floor(Q / 2^k), k = B - b, i.e. the top b bit planes;
 *  - LSB mask, Sec. 3.2.1 Eq. (lsb_masking): the masked weight keeps the
 *    stored n-bit scale, so the operand the layer multiplies is
 *    2^k * floor(Q / 2^k);
 *  - quantized linear, Sec. 3.1 Eq. (qalora): Y = Q(X) Q(W);
 *  - dequantisation, App. A.1.1-A.1.2: a product of per-tensor activation and
 *    per-output-channel weight scales (the 2^n/(2^n-1) weight factor folded
 *    into the channel scale, zero points zero);
 *  - stages, Sec. 3.2 (contiguous stages) and Sec. 4.1 (20 steps in four
 *    stages; four steps, one per stage), stage 0 the noisiest (App. D.1).
 *
 * Parity pins: every function here is checked by the CPU test suite against
 * an independent route (the paper's unsigned-code form of the mask applied
 * one bit at a time, a bitwise mask, hand-derived worked values, numpy's
 * int64 matmul at b = 8, an im2col convolution, a pure-Python brute force,
 * and the bit-plane identity).  No function is parity-unpinned.
 */
#include <stdint.h>
#include <stddef.h>
#include <math.h>
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORACLE_OK = 0, ORACLE_EBITS = 1, ORACLE_EOVERFLOW = 2, ORACLE_EDIM = 3 };

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of the following calls (the CPU baseline times one and all). */
void oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* floor(w / 2^k) toward minus infinity, by integer division and correction. */
static int64_t floor_div_pow2(int64_t w, int k)
{
    int64_t d = (int64_t)1 << k;
    int64_t q = w / d;              /* C truncates toward zero */
    if (w % d != 0 && w < 0)
        q -= 1;
    return q;
}

/* The masked operand: 2^k * floor(w / 2^k) with k = 8 - b. */
static int64_t masked_value(int64_t w, int b)
{
    int k = 8 - b;
    return ((int64_t)1 << k) * floor_div_pow2(w, k);
}

/* The operand at precision b (App. G.2 Eq. hw_rightshift), in the masked
 * form that keeps the stored scale (Sec. 3.2.1 Eq. lsb_masking). */
int oracle_mask(const int8_t *W, int64_t n, int b, int8_t *out)
{
    if (b < 1 || b > 8)
        return ORACLE_EBITS;
    for (int64_t i = 0; i < n; ++i)
        out[i] = (int8_t)masked_value(W[i], b);
    return ORACLE_OK;
}

/* Sec. 3.2 / Sec. 4.1: equal contiguous stages, s = floor(t * S / T). */
int oracle_stage_of_step(int t, int S, int T)
{
    if (S < 1 || T < 1 || S > T || t < 0 || t >= T)
        return -1;
    return (int)(((int64_t)t * S) / T);
}

/*
 * acc[m][n] = sum_k X[m][k] * (2^(8-b) * floor(W[n][k] / 2^(8-b)))
 * y[m][n]   = acc[m][n] * sx * sw[n] (+ bias[n])         (fp64)
 *
 * X int8 [M][K], W int8 [N][K] (output x input), acc int32 [M][N],
 * y fp64 [M][N]; bias may be NULL; acc or y may be NULL.
 * Returns ORACLE_EOVERFLOW if any |acc| >= 2^31 (acc then holds garbage).
 */
int oracle_masked_linear(const int8_t *X, const int8_t *W, double sx, const float *sw,
                         const float *bias, int64_t M, int64_t N, int64_t K, int b,
                         int32_t *acc, double *y)
{
    if (b < 1 || b > 8)
        return ORACLE_EBITS;
    if (M < 0 || N < 0 || K < 0)
        return ORACLE_EDIM;
    int overflow = 0;
#pragma omp parallel for schedule(static) reduction(| : overflow)
    for (int64_t m = 0; m < M; ++m) {
        for (int64_t n = 0; n < N; ++n) {
            int64_t s = 0;
            for (int64_t k = 0; k < K; ++k)
                s += (int64_t)X[m * K + k] * masked_value(W[n * K + k], b);
            if (s >= ((int64_t)1 << 31) || s < -((int64_t)1 << 31))
                overflow = 1;
            if (acc)
                acc[m * N + n] = (int32_t)s;
            if (y) {
                double v = (double)s * sx * (double)sw[n];
                if (bias)
                    v += (double)bias[n];
                y[m * N + n] = v;
            }
        }
    }
    return overflow ? ORACLE_EOVERFLOW : ORACLE_OK;
}

/*
 * Entries (rows[i], cols[i]) of the same product, one dot product each, for
 * sampled checks of outputs too large to recompute whole.  X is given as the
 * full [M][K] array or any [R][K] array addressed by rows[].
 */
int oracle_masked_linear_entries(const int8_t *X, const int8_t *W, double sx,
                                 const float *sw, const float *bias, int64_t K, int b,
                                 const int64_t *rows, const int64_t *cols, int64_t count,
                                 int32_t *acc, double *y)
{
    if (b < 1 || b > 8)
        return ORACLE_EBITS;
    int overflow = 0;
#pragma omp parallel for schedule(static) reduction(| : overflow)
    for (int64_t i = 0; i < count; ++i) {
        int64_t m = rows[i], n = cols[i];
        int64_t s = 0;
        for (int64_t k = 0; k < K; ++k)
            s += (int64_t)X[m * K + k] * masked_value(W[n * K + k], b);
        if (s >= ((int64_t)1 << 31) || s < -((int64_t)1 << 31))
            overflow = 1;
        acc[i] = (int32_t)s;
        double v = (double)s * sx * (double)sw[n];
        if (bias)
            v += (double)bias[n];
        y[i] = v;
    }
    return overflow ? ORACLE_EOVERFLOW : ORACLE_OK;
}

/*
 * Direct 3x3 convolution, stride 1, zero padding 1, NHWC, batch 1:
 * acc[h][w][co] = sum_{r,s,ci} X[h+r-1][w+s-1][ci] * Wb[co][r][s][ci].
 * Written as the convolution sum, not as a matrix product, so that the
 * (r, s, ci) ordering of a kernel's implicit GEMM is checked independently.
 */
int oracle_conv3x3(const int8_t *X, const int8_t *Wt, double sx, const float *sw,
                   const float *bias, int64_t H, int64_t Wd, int64_t Ci, int64_t Co, int b,
                   int32_t *acc, double *y)
{
    if (b < 1 || b > 8)
        return ORACLE_EBITS;
    int overflow = 0;
#pragma omp parallel for schedule(static) reduction(| : overflow)
    for (int64_t h = 0; h < H; ++h) {
        for (int64_t w = 0; w < Wd; ++w) {
            for (int64_t co = 0; co < Co; ++co) {
                int64_t s = 0;
                for (int64_t r = 0; r < 3; ++r) {
                    int64_t hh = h + r - 1;
                    if (hh < 0 || hh >= H)
                        continue;
                    for (int64_t q = 0; q < 3; ++q) {
                        int64_t ww = w + q - 1;
                        if (ww < 0 || ww >= Wd)
                            continue;
                        const int8_t *xp = X + (hh * Wd + ww) * Ci;
                        const int8_t *wp = Wt + ((co * 3 + r) * 3 + q) * Ci;
                        for (int64_t ci = 0; ci < Ci; ++ci)
                            s += (int64_t)xp[ci] * masked_value(wp[ci], b);
                    }
                }
                if (s >= ((int64_t)1 << 31) || s < -((int64_t)1 << 31))
                    overflow = 1;
                int64_t o = (h * Wd + w) * Co + co;
                if (acc)
                    acc[o] = (int32_t)s;
                if (y) {
                    double v = (double)s * sx * (double)sw[co];
                    if (bias)
                        v += (double)bias[co];
                    y[o] = v;
                }
            }
        }
    }
    return overflow ? ORACLE_EOVERFLOW : ORACLE_OK;
}

/*
 * Entries (pix[i], cols[i]) of the same convolution, pix = h*Wd + w, each
 * computed as its own convolution sum, for sampled checks of large layers.
 */
int oracle_conv3x3_entries(const int8_t *X, const int8_t *Wt, double sx, const float *sw,
                           const float *bias, int64_t H, int64_t Wd, int64_t Ci, int b,
                           const int64_t *pix, const int64_t *cols, int64_t count,
                           int32_t *acc, double *y)
{
    if (b < 1 || b > 8)
        return ORACLE_EBITS;
    int overflow = 0;
#pragma omp parallel for schedule(static) reduction(| : overflow)
    for (int64_t i = 0; i < count; ++i) {
        int64_t h = pix[i] / Wd, w = pix[i] % Wd, co = cols[i];
        int64_t s = 0;
        for (int64_t r = 0; r < 3; ++r) {
            int64_t hh = h + r - 1;
            if (hh < 0 || hh >= H)
                continue;
            for (int64_t q = 0; q < 3; ++q) {
                int64_t ww = w + q - 1;
                if (ww < 0 || ww >= Wd)
                    continue;
                const int8_t *xp = X + (hh * Wd + ww) * Ci;
                const int8_t *wp = Wt + ((co * 3 + r) * 3 + q) * Ci;
                for (int64_t ci = 0; ci < Ci; ++ci)
                    s += (int64_t)xp[ci] * masked_value(wp[ci], b);
            }
        }
        if (s >= ((int64_t)1 << 31) || s < -((int64_t)1 << 31))
            overflow = 1;
        acc[i] = (int32_t)s;
        double v = (double)s * sx * (double)sw[co];
        if (bias)
            v += (double)bias[co];
        y[i] = v;
    }
    return overflow ? ORACLE_EOVERFLOW : ORACLE_OK;
}

/*
 * Bit planes of the stored two's-complement weight (App. G.2: plane p is bit
 * p of the code, p = 0 the least significant).  Layout, in uint32 words:
 *   planes[nb][q][kb][r][w][f],  n = 32 nb + 16 f + r (r < 16),
 *   q = 7 - p (most significant plane first, so the top b planes of a
 *   32-channel block are one contiguous run), kb = j / 128.
 * Element j of row n, with e = j % 128, is sub-step s = e / 32, half
 * h = (e % 32) / 16, group i = (e % 16) / 4 and byte c = e % 4 of its
 * 16-element half; it goes to word w = 2 h + s / 2, at bit
 *   (8 c + g + p) mod 32,  g = 4 (s % 2) + i.
 * (A word holds one half's 16 elements of two sub-steps; plane p's word is
 * the plain byte-sliced word rotated left by p bits.)  NB = ceil(N / 32),
 * KB = ceil(K / 128); bits of channels past N and of codes past K are zero.
 * A storage layout of the same bits, not arithmetic.
 */
int oracle_pack_planes(const int8_t *W, int64_t N, int64_t K, uint32_t *planes)
{
    int64_t KB = (K + 127) / 128, NB = (N + 31) / 32;
    for (int64_t i = 0; i < NB * 8 * KB * 128; ++i)
        planes[i] = 0;
    for (int q = 0; q < 8; ++q) {
        int p = 7 - q;
        for (int64_t n = 0; n < N; ++n) {
            int64_t nb = n / 32, f = (n % 32) / 16, r = n % 16;
            for (int64_t j = 0; j < K; ++j) {
                uint32_t bit = ((uint32_t)(uint8_t)W[n * K + j] >> p) & 1u;
                int e = (int)(j % 128);
                int s = e / 32, h = (e % 32) / 16, i = (e % 16) / 4, c = e % 4;
                int w = 2 * h + s / 2, g = 4 * (s % 2) + i;
                int64_t word = (((nb * 8 + q) * KB + j / 128) * 16 + r) * 8 + 2 * w + f;
                planes[word] |= bit << ((8 * c + g + p) % 32);
            }
        }
    }
    return ORACLE_OK;
}

/*
 * The stored weight in the operand order of the int8 matrix instruction (a
 * storage layout of the same codes; the paper's one 8-bit buffer).  Element
 * W[n][k] goes to byte
 *   ((nb * KS + ks) * 64 + l) * 16 + (k % 16),
 *   nb = n / 32, ks = k / 32, l = n % 32 + 32 * ((k % 32) / 16),
 * with KS = 4 * ceil(K / 128); the buffer holds 32 * ceil(N / 32) rows by
 * 128 * ceil(K / 128) columns' worth of bytes, zero where no element lands.
 */
int oracle_pack_weights(const int8_t *W, int64_t N, int64_t K, int8_t *packed)
{
    int64_t KS = 4 * ((K + 127) / 128);
    int64_t bytes = 32 * ((N + 31) / 32) * 128 * ((K + 127) / 128);
    for (int64_t i = 0; i < bytes; ++i)
        packed[i] = 0;
    for (int64_t n = 0; n < N; ++n)
        for (int64_t k = 0; k < K; ++k) {
            int64_t nb = n / 32, ks = k / 32;
            int64_t l = n % 32 + 32 * ((k % 32) / 16);
            packed[((nb * KS + ks) * 64 + l) * 16 + k % 16] = W[n * K + k];
        }
    return ORACLE_OK;
}

/*
 * Activation quantizer of App. A.1.2 (Eqs. act_quant, act_scale), n = 8,
 * per tensor:
 *   alpha = (max(x) - min(x)) / (2^n - 1),   z = -min(x) / alpha,
 *   Q = clamp(round_to_nearest(x / alpha + z), 0, 2^n - 1).
 * z is kept real, as printed.  Each operation is one IEEE single-precision
 * operation in this order (the subtraction, the divisions, then the
 * addition), rounding ties to even: the precision the kernel decides the
 * codes in.  When max == min the scale is undefined; alpha = 1 and z = -min
 * are taken, so every code is 0 and dequantises to min exactly.
 * x must be finite.
 */
int oracle_act_quant(const float *x, int64_t n, float *alpha_out, float *z_out, uint8_t *q)
{
    if (n <= 0)
        return ORACLE_EDIM;
    float mn = x[0], mx = x[0];
    for (int64_t i = 1; i < n; ++i) {
        if (x[i] < mn)
            mn = x[i];
        if (x[i] > mx)
            mx = x[i];
    }
    float alpha, z;
    if (mx == mn) {
        alpha = 1.0f;
        z = -mn;
    } else {
        float range = mx - mn;
        alpha = range / 255.0f;
        z = -mn / alpha;
    }
    for (int64_t i = 0; i < n; ++i) {
        float t = x[i] / alpha;
        t = t + z;
        float r = rintf(t);
        if (r < 0.0f)
            r = 0.0f;
        if (r > 255.0f)
            r = 255.0f;
        q[i] = (uint8_t)r;
    }
    *alpha_out = alpha;
    *z_out = z;
    return ORACLE_OK;
}

/*
 * Per-output-channel sums of the masked weight at every precision, for the
 * zero-point term of an asymmetric activation:
 *   colsum[b-1][n] = sum_k 2^(8-b) floor(W[n][k] / 2^(8-b)),  b = 1..8.
 */
int oracle_weight_colsums(const int8_t *W, int64_t N, int64_t K, int32_t *colsum)
{
    if (N < 0 || K < 0)
        return ORACLE_EDIM;
    for (int b = 1; b <= 8; ++b)
        for (int64_t n = 0; n < N; ++n) {
            int64_t s = 0;
            for (int64_t k = 0; k < K; ++k)
                s += masked_value(W[n * K + k], b);
            colsum[(b - 1) * N + n] = (int32_t)s;
        }
    return ORACLE_OK;
}

/*
 * The layer on asymmetric activation codes Q (App. A.1.2: x_hat =
 * alpha (Q - z)) and the masked weight (per-channel scale sw):
 *   y[m][n]   = sum_k alpha (Q[m][k] - z) * sw[n] W_b[n][k]  (+ bias[n])   fp64,
 *               the definition, summed in ascending k;
 *   acc[m][n] = sum_k (Q[m][k] - 128) W_b[n][k]                          int32,
 *               the integer product of the signed codes Q - 128 that the
 *               int8 matrix instruction consumes.
 * Q uint8 [M][K]; other arguments as oracle_masked_linear.
 */
int oracle_masked_linear_asym(const uint8_t *Q, const int8_t *W, double alpha, double z,
                              const float *sw, const float *bias, int64_t M, int64_t N,
                              int64_t K, int b, int32_t *acc, double *y)
{
    if (b < 1 || b > 8)
        return ORACLE_EBITS;
    if (M < 0 || N < 0 || K < 0)
        return ORACLE_EDIM;
    int overflow = 0;
#pragma omp parallel for schedule(static) reduction(| : overflow)
    for (int64_t m = 0; m < M; ++m) {
        for (int64_t n = 0; n < N; ++n) {
            int64_t s = 0;
            double v = 0.0;
            for (int64_t k = 0; k < K; ++k) {
                int64_t w = masked_value(W[n * K + k], b);
                s += ((int64_t)Q[m * K + k] - 128) * w;
                v += alpha * ((double)Q[m * K + k] - z) * (double)sw[n] * (double)w;
            }
            if (s >= ((int64_t)1 << 31) || s < -((int64_t)1 << 31))
                overflow = 1;
            if (acc)
                acc[m * N + n] = (int32_t)s;
            if (y) {
                if (bias)
                    v += (double)bias[n];
                y[m * N + n] = v;
            }
        }
    }
    return overflow ? ORACLE_EOVERFLOW : ORACLE_OK;
}

/* Entries (rows[i], cols[i]) of oracle_masked_linear_asym, one dot product
 * each (rows index Q, cols index W, sw and bias). */
int oracle_masked_linear_asym_entries(const uint8_t *Q, const int8_t *W, double alpha, double z,
                                      const float *sw, const float *bias, int64_t K, int b,
                                      const int64_t *rows, const int64_t *cols, int64_t count,
                                      int32_t *acc, double *y)
{
    if (b < 1 || b > 8)
        return ORACLE_EBITS;
    int overflow = 0;
#pragma omp parallel for schedule(static) reduction(| : overflow)
    for (int64_t i = 0; i < count; ++i) {
        const int64_t m = rows[i], n = cols[i];
        int64_t s = 0;
        double v = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            int64_t w = masked_value(W[n * K + k], b);
            s += ((int64_t)Q[m * K + k] - 128) * w;
            v += alpha * ((double)Q[m * K + k] - z) * (double)sw[n] * (double)w;
        }
        if (s >= ((int64_t)1 << 31) || s < -((int64_t)1 << 31))
            overflow = 1;
        acc[i] = (int32_t)s;
        if (bias)
            v += (double)bias[n];
        y[i] = v;
    }
    return overflow ? ORACLE_EOVERFLOW : ORACLE_OK;
}

/*
 * Weight quantizer of App. A.1.1 (Eqs. weight_quant, weight_scale,
 * weight_dequant), n bits, one scale and zero point per output channel
 * (row of W [N][K]):
 *   alpha = (max(w) - min(w)) / 2^n,   z = -min(w) / alpha,
 *   Q = clamp(floor(w / alpha + z), 0, 2^n - 1),
 *   w_hat = 2^n / (2^n - 1) * alpha * (Q - z),
 * and sw = alpha * 2^n / (2^n - 1), the per-channel factor of w_hat, so that
 * w_hat = sw * (Q - z).  Each operation is one IEEE single-precision
 * operation in this order, as for the activation quantizer; sw is
 * (alpha * 2^n) / (2^n - 1), the product exact.  A constant row takes
 * alpha = 1, z = -min (every code 0).  W must be finite.
 */
int oracle_weight_quant(const float *W, int64_t N, int64_t K, int nbits, uint8_t *Q,
                        float *alpha_out, float *z_out, float *sw_out)
{
    if (N < 0 || K <= 0 || nbits < 1 || nbits > 8)
        return ORACLE_EDIM;
    const float levels = (float)(1 << nbits);
    const float top = levels - 1.0f;
    for (int64_t n = 0; n < N; ++n) {
        const float *w = W + n * K;
        float mn = w[0], mx = w[0];
        for (int64_t k = 1; k < K; ++k) {
            if (w[k] < mn)
                mn = w[k];
            if (w[k] > mx)
                mx = w[k];
        }
        float alpha, z;
        if (mx == mn) {
            alpha = 1.0f;
            z = -mn;
        } else {
            float range = mx - mn;
            alpha = range / levels;
            z = -mn / alpha;
        }
        for (int64_t k = 0; k < K; ++k) {
            float t = w[k] / alpha;
            t = t + z;
            float f = floorf(t);
            if (f < 0.0f)
                f = 0.0f;
            if (f > top)
                f = top;
            Q[n * K + k] = (uint8_t)f;
        }
        float scaled = alpha * levels;
        alpha_out[n] = alpha;
        z_out[n] = z;
        sw_out[n] = scaled / top;
    }
    return ORACLE_OK;
}

/*
 * The layer with both operands dequantised (App. A.1), in fp64 from the
 * definitions, summed in ascending k:
 *   y[m][n] = sum_k x_hat[m][k] * w_hat_b[n][k]  (+ bias[n]),
 *   x_hat = sx * X                     (symmetric codes X, asym_x = 0), or
 *   x_hat = ax * ((X + 128) - zx)      (asymmetric codes Q = X + 128),
 *   w_hat_b = sw[n] * W_b              (zw == NULL: zero point 0), or
 *   w_hat_b = sw[n] * ((W_b + 128) - zw[n])   (the masked code Q_b = W_b + 128
 *                                              with the channel's real zero point);
 *   acc[m][n] = sum_k X[m][k] * W_b[n][k]  int32, the product of the signed
 *   codes the int8 matrix instruction consumes.
 * X, W int8 signed codes; other arguments as oracle_masked_linear.
 */
static double xhat_of(int8_t x, int asym_x, double sx, double ax, double zx)
{
    return asym_x ? ax * (((double)x + 128.0) - zx) : sx * (double)x;
}

int oracle_layer_dequant(const int8_t *X, int asym_x, double sx, double ax, double zx,
                         const int8_t *W, const float *sw, const float *zw, const float *bias,
                         int64_t M, int64_t N, int64_t K, int b, int32_t *acc, double *y)
{
    if (b < 1 || b > 8)
        return ORACLE_EBITS;
    if (M < 0 || N < 0 || K < 0)
        return ORACLE_EDIM;
    int overflow = 0;
#pragma omp parallel for schedule(static) reduction(| : overflow)
    for (int64_t m = 0; m < M; ++m) {
        for (int64_t n = 0; n < N; ++n) {
            int64_t s = 0;
            double v = 0.0;
            for (int64_t k = 0; k < K; ++k) {
                const int64_t wb = masked_value(W[n * K + k], b);
                const int8_t x = X[m * K + k];
                s += (int64_t)x * wb;
                const double what = zw ? (double)sw[n] * (((double)wb + 128.0) - (double)zw[n])
                                       : (double)sw[n] * (double)wb;
                v += xhat_of(x, asym_x, sx, ax, zx) * what;
            }
            if (s >= ((int64_t)1 << 31) || s < -((int64_t)1 << 31))
                overflow = 1;
            if (acc)
                acc[m * N + n] = (int32_t)s;
            if (y)
                y[m * N + n] = v + (bias ? (double)bias[n] : 0.0);
        }
    }
    return overflow ? ORACLE_EOVERFLOW : ORACLE_OK;
}

/* Entries (rows[i], cols[i]) of oracle_layer_dequant. */
int oracle_layer_dequant_entries(const int8_t *X, int asym_x, double sx, double ax, double zx,
                                 const int8_t *W, const float *sw, const float *zw,
                                 const float *bias, int64_t K, int b, const int64_t *rows,
                                 const int64_t *cols, int64_t count, int32_t *acc, double *y)
{
    if (b < 1 || b > 8)
        return ORACLE_EBITS;
    int overflow = 0;
#pragma omp parallel for schedule(static) reduction(| : overflow)
    for (int64_t i = 0; i < count; ++i) {
        const int64_t m = rows[i], n = cols[i];
        int64_t s = 0;
        double v = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            const int64_t wb = masked_value(W[n * K + k], b);
            const int8_t x = X[m * K + k];
            s += (int64_t)x * wb;
            const double what = zw ? (double)sw[n] * (((double)wb + 128.0) - (double)zw[n])
                                   : (double)sw[n] * (double)wb;
            v += xhat_of(x, asym_x, sx, ax, zx) * what;
        }
        if (s >= ((int64_t)1 << 31) || s < -((int64_t)1 << 31))
            overflow = 1;
        acc[i] = (int32_t)s;
        y[i] = v + (bias ? (double)bias[n] : 0.0);
    }
    return overflow ? ORACLE_EOVERFLOW : ORACLE_OK;
}
