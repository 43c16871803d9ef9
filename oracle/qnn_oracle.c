/*
 * qnn_oracle.c -- CPU oracle for quantized conv2d / depthwise conv2d / dense
 * with requantize and add (TEST INFRASTRUCTURE ONLY).
 *
 * Only the tests, the smoke check and the CPU-baseline leg of the benchmark
 * may load this library.  The product path (the HIP library) shares no code,
 * header, table or helper with it; neither includes nor links the other.
 *
 * Everything here is the plain definition written out as naive int64 loop
 * nests, in the order the paper states it, with no blocking or fusion:
 *
 *   - Quantized tensor semantics, Eq. (1): real = scale * (Q - zp).
 *   - Quantized conv2d, Eq. (2)/(3): the integer accumulator is the sum over
 *     (c, r, s) of (Q_A - zp_A) * (Q_B - zp_B), i.e. the product form that the
 *     four-term expansion of Eq. (3) rearranges.  Padding of the input uses
 *     the input zero point (Sec. III-B, "QNN Convolution Operator"), so
 *     padded taps contribute exactly zero.  The generalisation to stride,
 *     asymmetric padding, dilation and per-output-channel weight zero points
 *     is the obvious one (the paper writes Eq. (3) for stride 1, no padding).
 *   - Bias (TFLite conv = qnn.conv2d -> bias_add -> clip -> requantize,
 *     Sec. III-A, Fig. 2): int32 with implied scale s_x * s_w[k], zero point 0,
 *     added to the accumulator before requantize.
 *   - Requantize, Eq. (5), with the fixed-point multiplier of Sec. III-B:
 *     M = s_in / s_out as binary64, M = f * 2^e with f in [0.5, 1),
 *     mult = floor(f * 2^31 + 1/2) in [2^30, 2^31], renormalised to 2^30 with
 *     e + 1 when it reaches 2^31, shift n = 31 - e; the result is
 *     round(v * mult / 2^n) under the selected rounding, then + zp_out, then
 *     saturation to the output range intersected with the activation clamp.
 *     The paper leaves the rounding open to the framework; three are
 *     defined: HALF_UP (ties toward +infinity), HALF_AWAY (ties away from
 *     zero) and TWO_STAGE, the integer-only form of Jacob et al. (the
 *     paper's reference for pre-quantized TFLite models): for n >= 31 the
 *     product is first divided by 2^31 and rounded half up (a rounding
 *     high multiply), that result then divided by 2^(n - 31) and rounded
 *     half away from zero (a rounding right shift); for n < 31 a single
 *     half-up rounding.
 *   - qnn.add: each input is requantized to the output scale (without its
 *     own output zero point), the two are added, then zp_out and the clamp.
 *   - Quantized pooling, Eq. (4): input and output share one scale and
 *     zero point, so the quantized output is the pooled quantized input.
 *     Average: the sum of the window's cells (wide integers, no overflow)
 *     divided by the cell count and rounded to the nearest integer, ties by
 *     the selected rounding (HALF_UP or HALF_AWAY; the paper asks for care
 *     with this rounding but does not fix it).  Cells outside the input are
 *     either left out of sum and count, or counted with the zero point as
 *     their value (a real zero).  Max: the largest in-input cell (scale > 0
 *     makes max commute with dequantization).
 *
 * Parity pins (checked by the CPU test suite, not by this file): exact
 * rational dequantize identity of Eq. (1)/(2), the four-term expansion of
 * Eq. (3), float64 library convolution, closed-form fixtures, and exact
 * rational rounding for the fixed-point requantize.
 */
#include <stdint.h>
#include <stdlib.h>
#include <math.h>
#include <omp.h>

#define ORACLE_U8 0
#define ORACLE_I8 1
#define ORACLE_I32 2

#define ORACLE_HALF_UP 0
#define ORACLE_HALF_AWAY 1
#define ORACLE_TWO_STAGE 2

/* Read element i of a quantized tensor of dtype dt, widened to int64. */
static int64_t q_load(const void *p, int dt, int64_t i)
{
    if (dt == ORACLE_U8)
        return ((const uint8_t *)p)[i];
    if (dt == ORACLE_I8)
        return ((const int8_t *)p)[i];
    return ((const int32_t *)p)[i];
}

static void q_store(void *p, int dt, int64_t i, int64_t v)
{
    if (dt == ORACLE_U8)
        ((uint8_t *)p)[i] = (uint8_t)v;
    else if (dt == ORACLE_I8)
        ((int8_t *)p)[i] = (int8_t)v;
    else
        ((int32_t *)p)[i] = (int32_t)v;
}

static int64_t dtype_min(int dt)
{
    if (dt == ORACLE_U8) return 0;
    if (dt == ORACLE_I8) return -128;
    return -2147483648LL;
}

static int64_t dtype_max(int dt)
{
    if (dt == ORACLE_U8) return 255;
    if (dt == ORACLE_I8) return 127;
    return 2147483647LL;
}

/* Floor of x / 2^n for n in [0, 62], written as a plain division so the
 * rounding direction is visible: C division truncates toward zero, so a
 * negative quotient with a remainder is moved down by one. */
static int64_t floor_div_pow2(int64_t x, int n)
{
    int64_t d = (int64_t)1 << n;
    int64_t q = x / d;
    if ((x % d) != 0 && x < 0)
        q -= 1;
    return q;
}

/*
 * Fixed-point form of a real multiplier M >= 0 (Eq. (5) with the fixed-point
 * proxy of Sec. III-B).  On success returns 0 and sets *mult, *shift such
 * that M ~= mult * 2^-shift, mult in [2^30, 2^31) and shift >= 1; M == 0 gives
 * mult = 0, shift = 1.  Returns -1 when M is negative, not finite, or so
 * large that the shift would fall below 1.
 */
int oracle_quantize_multiplier(double M, int32_t *mult, int32_t *shift)
{
    if (!(M >= 0.0) || isinf(M))
        return -1;
    if (M == 0.0) {
        *mult = 0;
        *shift = 1;
        return 0;
    }
    int e = 0;
    double f = frexp(M, &e);            /* M = f * 2^e, 0.5 <= f < 1 */
    double scaled = ldexp(f, 31);       /* exact: power-of-two scaling */
    int64_t q = (int64_t)floor(scaled + 0.5); /* exact in binary64 */
    if (q == ((int64_t)1 << 31)) {
        q = (int64_t)1 << 30;
        e += 1;
    }
    int n = 31 - e;
    if (n < 1)
        return -1;
    *mult = (int32_t)q;
    *shift = n;
    return 0;
}

/* Real multiplier of a requantize from scale s_in to scale s_out.  The
 * product of two binary32 values is exact in binary64, so for a conv the
 * caller passes s_in = (double)s_x * (double)s_w[k] and only the division
 * rounds. */
static double real_multiplier(double s_in, double s_out)
{
    return s_in / s_out;
}

/* round(v * mult / 2^shift) under the given rounding; mult == 0 gives 0. */
int64_t oracle_round_mul_shift(int64_t v, int32_t mult, int32_t shift, int rounding)
{
    if (mult == 0)
        return 0;
    int64_t p = v * (int64_t)mult;
    if (shift >= 63)
        return 0; /* |p| < 2^62, so |p| / 2^shift < 1/2 */
    if (rounding == ORACLE_TWO_STAGE && shift >= 31) {
        /* stage 1: p / 2^31 rounded half up */
        int64_t x1 = floor_div_pow2(p + ((int64_t)1 << 30), 31);
        int e = shift - 31;
        if (e == 0)
            return x1;
        /* stage 2: x1 / 2^e rounded half away from zero */
        int64_t m = x1 < 0 ? -x1 : x1;
        int64_t r = floor_div_pow2(m + ((int64_t)1 << (e - 1)), e);
        return x1 < 0 ? -r : r;
    }
    int64_t half = (int64_t)1 << (shift - 1);
    if (rounding == ORACLE_HALF_UP || rounding == ORACLE_TWO_STAGE)
        return floor_div_pow2(p + half, shift);
    /* HALF_AWAY: round the magnitude half up, then restore the sign */
    int64_t a = p < 0 ? -p : p;
    int64_t t = floor_div_pow2(a + half, shift);
    return p < 0 ? -t : t;
}

static int64_t clamp64(int64_t v, int64_t lo, int64_t hi)
{
    return v < lo ? lo : (v > hi ? hi : v);
}

/*
 * Requantize one value v (already zero-point adjusted) with multiplier M
 * into dtype yt: Eq. (5) plus saturation.  lo/hi are the activation clamp in
 * the output Q domain; the effective range is their intersection with the
 * dtype range.  Returns -1 for an invalid multiplier.
 */
static int requantize_one(int64_t v, double M, int32_t zp_out, int yt,
                          int64_t lo, int64_t hi, int rounding, int64_t *out)
{
    int32_t mult, shift;
    /* the domain of the fixed-point product: |v| <= 2^31 keeps |v*mult| < 2^62 */
    if (v > ((int64_t)1 << 31) || v < -((int64_t)1 << 31))
        return -1;
    if (oracle_quantize_multiplier(M, &mult, &shift) != 0)
        return -1;
    int64_t t = oracle_round_mul_shift(v, mult, shift, rounding);
    int64_t l = lo > dtype_min(yt) ? lo : dtype_min(yt);
    int64_t h = hi < dtype_max(yt) ? hi : dtype_max(yt);
    *out = clamp64(t + zp_out, l, h);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Accumulators                                                             */
/* ------------------------------------------------------------------------ */

static int64_t out_dim(int64_t in, int64_t pad_a, int64_t pad_b, int64_t dil,
                       int64_t k, int64_t stride)
{
    return (in + pad_a + pad_b - dil * (k - 1) - 1) / stride + 1;
}

typedef struct {
    int64_t N, H, W, C;      /* input NHWC */
    int64_t K, R, S;         /* output channels, filter height/width */
    int64_t sh, sw, pt, pl, pb, pr, dh, dw;
    int64_t Ho, Wo;
} conv_geom;

static conv_geom make_geom(const int32_t *shape /* N,H,W,C,K,R,S */,
                           const int32_t *cp /* sh,sw,pt,pl,pb,pr,dh,dw */)
{
    conv_geom g;
    g.N = shape[0]; g.H = shape[1]; g.W = shape[2]; g.C = shape[3];
    g.K = shape[4]; g.R = shape[5]; g.S = shape[6];
    g.sh = cp[0]; g.sw = cp[1]; g.pt = cp[2]; g.pl = cp[3];
    g.pb = cp[4]; g.pr = cp[5]; g.dh = cp[6]; g.dw = cp[7];
    g.Ho = out_dim(g.H, g.pt, g.pb, g.dh, g.R, g.sh);
    g.Wo = out_dim(g.W, g.pl, g.pr, g.dw, g.S, g.sw);
    return g;
}

/*
 * Input value at (n, ih, iw, c) with zero-point padding: inside the image
 * it is Q_x, outside it is zp_x (real 0.0 is represented by the zero point).
 */
static int64_t x_padded(const void *x, int xt, const conv_geom *g, int64_t n,
                        int64_t ih, int64_t iw, int64_t c, int64_t zp_x)
{
    if (ih < 0 || ih >= g->H || iw < 0 || iw >= g->W)
        return zp_x;
    return q_load(x, xt, ((n * g->H + ih) * g->W + iw) * g->C + c);
}

/*
 * One conv2d accumulator (Eq. (2)/(3) in product form) plus bias:
 *   acc = bias[k] + sum_{r,s,c} (x~[n, oh*sh + r*dh - pt, ow*sw + s*dw - pl, c]
 *                                 - zp_x) * (w[k,r,s,c] - zp_w[k])
 * with w in OHWI order, of dtype wt: int8, or uint8 as in pre-quantized
 * models whose weights are asymmetric uint8 (the weight zero point is then
 * in [0, 255]).
 */
static int64_t conv_acc_one(const void *x, int xt, int64_t zp_x, const void *w, int wt,
                            const int32_t *zp_w, const int32_t *bias,
                            const conv_geom *g, int64_t n, int64_t oh,
                            int64_t ow, int64_t k)
{
    int64_t acc = 0;
    for (int64_t r = 0; r < g->R; ++r)
        for (int64_t s = 0; s < g->S; ++s)
            for (int64_t c = 0; c < g->C; ++c) {
                int64_t ih = oh * g->sh + r * g->dh - g->pt;
                int64_t iw = ow * g->sw + s * g->dw - g->pl;
                int64_t a = x_padded(x, xt, g, n, ih, iw, c, zp_x) - zp_x;
                int64_t b = q_load(w, wt, ((k * g->R + r) * g->S + s) * g->C + c) - zp_w[k];
                acc += a * b;
            }
    if (bias)
        acc += bias[k];
    return acc;
}

/* Depthwise (channel multiplier 1): w is [R][S][C]. */
static int64_t dw_acc_one(const void *x, int xt, int64_t zp_x, const void *w, int wt,
                          const int32_t *zp_w, const int32_t *bias,
                          const conv_geom *g, int64_t n, int64_t oh,
                          int64_t ow, int64_t c)
{
    int64_t acc = 0;
    for (int64_t r = 0; r < g->R; ++r)
        for (int64_t s = 0; s < g->S; ++s) {
            int64_t ih = oh * g->sh + r * g->dh - g->pt;
            int64_t iw = ow * g->sw + s * g->dw - g->pl;
            int64_t a = x_padded(x, xt, g, n, ih, iw, c, zp_x) - zp_x;
            int64_t b = q_load(w, wt, (r * g->S + s) * g->C + c) - zp_w[c];
            acc += a * b;
        }
    if (bias)
        acc += bias[c];
    return acc;
}

/* Output spatial size for the given shape and conv params. */
void oracle_conv_out_hw(const int32_t *shape, const int32_t *cp, int64_t *ho, int64_t *wo)
{
    conv_geom g = make_geom(shape, cp);
    *ho = g.Ho;
    *wo = g.Wo;
}

/*
 * Full conv2d accumulator tensor acc[n][oh][ow][k] (int64), including bias.
 * depthwise != 0 selects the channel-multiplier-1 depthwise form, where
 * shape[4] (K) must equal C and w is [R][S][C].
 */
void oracle_conv2d_acc(const void *x, int32_t xt, int32_t zp_x, const void *w, int32_t wt,
                       const int32_t *zp_w, const int32_t *bias,
                       const int32_t *shape, const int32_t *cp, int32_t depthwise,
                       int64_t *acc)
{
    conv_geom g = make_geom(shape, cp);
    int64_t rows = g.N * g.Ho;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t nr = 0; nr < rows; ++nr) {
        int64_t n = nr / g.Ho, oh = nr % g.Ho;
        for (int64_t ow = 0; ow < g.Wo; ++ow)
            for (int64_t k = 0; k < g.K; ++k) {
                int64_t m = (n * g.Ho + oh) * g.Wo + ow;
                acc[m * g.K + k] = depthwise
                    ? dw_acc_one(x, xt, zp_x, w, wt, zp_w, bias, &g, n, oh, ow, k)
                    : conv_acc_one(x, xt, zp_x, w, wt, zp_w, bias, &g, n, oh, ow, k);
            }
    }
}

/* Accumulators at selected flat output indices idx = m * K + k only. */
void oracle_conv2d_acc_points(const void *x, int32_t xt, int32_t zp_x, const void *w, int32_t wt,
                              const int32_t *zp_w, const int32_t *bias,
                              const int32_t *shape, const int32_t *cp, int32_t depthwise,
                              const int64_t *idx, int64_t npts, int64_t *acc)
{
    conv_geom g = make_geom(shape, cp);
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t i = 0; i < npts; ++i) {
        int64_t m = idx[i] / g.K, k = idx[i] % g.K;
        int64_t ow = m % g.Wo, oh = (m / g.Wo) % g.Ho, n = m / (g.Wo * g.Ho);
        acc[i] = depthwise
            ? dw_acc_one(x, xt, zp_x, w, wt, zp_w, bias, &g, n, oh, ow, k)
            : conv_acc_one(x, xt, zp_x, w, wt, zp_w, bias, &g, n, oh, ow, k);
    }
}

/* Dense: acc[m][j] = bias[j] + sum_k (x[m,k] - zp_x) * (w[j,k] - zp_w[j]). */
void oracle_dense_acc(const void *x, int32_t xt, int32_t zp_x, const void *w, int32_t wt,
                      const int32_t *zp_w, const int32_t *bias, int64_t M,
                      int64_t Kd, int64_t Nd, int64_t *acc)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t j = 0; j < Nd; ++j) {
            int64_t a = 0;
            for (int64_t k = 0; k < Kd; ++k)
                a += (q_load(x, xt, m * Kd + k) - zp_x) *
                     (q_load(w, wt, j * Kd + k) - zp_w[j]);
            if (bias)
                a += bias[j];
            acc[m * Nd + j] = a;
        }
}

/* ------------------------------------------------------------------------ */
/* Requantize                                                               */
/* ------------------------------------------------------------------------ */

/*
 * Requantize accumulators of a conv / dense output with K channels on the
 * innermost axis: M_k = (s_x * s_w[k]) / s_y with s_w per channel (nw == K)
 * or per tensor (nw == 1).  Output element (m, k) is stored at
 * y[m * y_ldc + y_coff + k].  Returns 0, or -1 on an invalid multiplier.
 */
int oracle_requantize_acc(const int64_t *acc, int64_t Mrows, int64_t K,
                          float s_x, const float *s_w, int32_t nw, float s_y,
                          int32_t zp_y, int32_t yt, int64_t lo, int64_t hi,
                          int32_t rounding, void *y, int64_t y_ldc, int64_t y_coff)
{
    int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
    for (int64_t m = 0; m < Mrows; ++m)
        for (int64_t k = 0; k < K; ++k) {
            double sw = (double)s_w[nw == 1 ? 0 : k];
            double Mk = real_multiplier((double)s_x * sw, (double)s_y);
            int64_t out;
            if (requantize_one(acc[m * K + k], Mk, zp_y, yt, lo, hi, rounding, &out)) {
                bad = 1;
                continue;
            }
            q_store(y, yt, m * y_ldc + y_coff + k, out);
        }
    return bad ? -1 : 0;
}

/* Same, for a list of (flat index, accumulator) points; writes out[i]. */
int oracle_requantize_points(const int64_t *acc, const int64_t *idx, int64_t npts,
                             int64_t K, float s_x, const float *s_w, int32_t nw,
                             float s_y, int32_t zp_y, int32_t yt, int64_t lo,
                             int64_t hi, int32_t rounding, int64_t *out)
{
    int bad = 0;
    for (int64_t i = 0; i < npts; ++i) {
        int64_t k = idx[i] % K;
        double sw = (double)s_w[nw == 1 ? 0 : k];
        double Mk = real_multiplier((double)s_x * sw, (double)s_y);
        if (requantize_one(acc[i], Mk, zp_y, yt, lo, hi, rounding, &out[i]))
            bad = 1;
    }
    return bad ? -1 : 0;
}

/*
 * Standalone requantize (Eq. (5)) of `count` values of dtype xt whose
 * innermost axis has `channels` entries.  Input and output qparams are per
 * tensor (n == 1) or per channel (n == channels).
 *   y = clamp(zp_out[c] + round((q - zp_in[c]) * s_in[c] / s_out[c]), lo, hi)
 */
int oracle_requantize(const void *x, int32_t xt, int64_t count, int64_t channels,
                      const float *s_in, const int32_t *zp_in, int32_t n_in,
                      const float *s_out, const int32_t *zp_out, int32_t n_out,
                      int32_t yt, int64_t lo, int64_t hi, int32_t rounding, void *y)
{
    int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
    for (int64_t i = 0; i < count; ++i) {
        int64_t c = i % channels;
        int64_t ci = n_in == 1 ? 0 : c, co = n_out == 1 ? 0 : c;
        double M = real_multiplier((double)s_in[ci], (double)s_out[co]);
        int64_t out;
        if (requantize_one(q_load(x, xt, i) - zp_in[ci], M, zp_out[co], yt, lo, hi,
                           rounding, &out)) {
            bad = 1;
            continue;
        }
        q_store(y, yt, i, out);
    }
    return bad ? -1 : 0;
}

/*
 * qnn.add: y = clamp(zp_o + round((a - zp_a) * s_a / s_o)
 *                         + round((b - zp_b) * s_b / s_o), lo, hi)
 */
int oracle_add(const void *a, int32_t at, float s_a, int32_t zp_a,
               const void *b, int32_t bt, float s_b, int32_t zp_b,
               int64_t count, float s_o, int32_t zp_o, int32_t yt,
               int64_t lo, int64_t hi, int32_t rounding, void *y)
{
    int32_t ma, na, mb, nb;
    if (oracle_quantize_multiplier(real_multiplier(s_a, s_o), &ma, &na) ||
        oracle_quantize_multiplier(real_multiplier(s_b, s_o), &mb, &nb))
        return -1;
    int64_t l = lo > dtype_min(yt) ? lo : dtype_min(yt);
    int64_t h = hi < dtype_max(yt) ? hi : dtype_max(yt);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i) {
        int64_t ta = oracle_round_mul_shift(q_load(a, at, i) - zp_a, ma, na, rounding);
        int64_t tb = oracle_round_mul_shift(q_load(b, bt, i) - zp_b, mb, nb, rounding);
        q_store(y, yt, i, clamp64(zp_o + ta + tb, l, h));
    }
    return 0;
}

/* floor(a / b) for b > 0. */
static int64_t floor_div(int64_t a, int64_t b)
{
    return a >= 0 ? a / b : -((-a + b - 1) / b);
}

/* The integer nearest to sum / count (count > 0), ties toward +infinity
 * (HALF_UP) or away from zero (HALF_AWAY): floor((2*sum + count) / (2*count)),
 * with the magnitude rounded and the sign restored for HALF_AWAY. */
static int64_t round_div(int64_t sum, int64_t count, int rounding)
{
    if (rounding == ORACLE_HALF_AWAY) {
        const int64_t m = floor_div(2 * (sum < 0 ? -sum : sum) + count, 2 * count);
        return sum < 0 ? -m : m;
    }
    return floor_div(2 * sum + count, 2 * count);
}

/*
 * Quantized pool2d, Eq. (4).  shape = N,H,W,C,R,S; pp = stride_h, stride_w,
 * pad_top, pad_left, pad_bottom, pad_right; mode 0 average, 1 max;
 * count_pad 1 counts padded cells as holding zp.  x and y are NHWC of dtype
 * xt; Ho = (H + pt + pb - R) / stride_h + 1, likewise Wo.  Returns -1 when a
 * window holds no cell of the input.
 */
int oracle_pool2d(const void *x, int32_t xt, const int32_t *shape, const int32_t *pp, int32_t mode,
                  int32_t count_pad, int32_t zp, int32_t rounding, void *y)
{
    const int64_t N = shape[0], H = shape[1], W = shape[2], C = shape[3], R = shape[4], S = shape[5];
    const int64_t sh = pp[0], sw = pp[1], pt = pp[2], pl = pp[3], pb = pp[4], pr = pp[5];
    const int64_t Ho = (H + pt + pb - R) / sh + 1, Wo = (W + pl + pr - S) / sw + 1;
    int bad = 0;
#pragma omp parallel for collapse(2) reduction(| : bad)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t oh = 0; oh < Ho; ++oh)
            for (int64_t ow = 0; ow < Wo; ++ow)
                for (int64_t c = 0; c < C; ++c) {
                    int64_t sum = 0, count = 0, best = 0, seen = 0;
                    for (int64_t r = 0; r < R; ++r)
                        for (int64_t t = 0; t < S; ++t) {
                            const int64_t h = oh * sh - pt + r, w = ow * sw - pl + t;
                            if (h < 0 || h >= H || w < 0 || w >= W) {
                                if (count_pad) {
                                    sum += zp;
                                    ++count;
                                }
                                continue;
                            }
                            const int64_t v = q_load(x, xt, ((n * H + h) * W + w) * C + c);
                            sum += v;
                            ++count;
                            if (!seen || v > best)
                                best = v;
                            seen = 1;
                        }
                    if (!seen) {
                        bad = 1;
                        continue;
                    }
                    q_store(y, xt, ((n * Ho + oh) * Wo + ow) * C + c,
                            mode == 1 ? best : round_div(sum, count, rounding));
                }
    return bad ? -1 : 0;
}

/* Requantize of a single zero-point adjusted value v with real multiplier M
 * (exported for the exact-rational tests). */
int oracle_requantize_value(int64_t v, double M, int32_t zp_out, int32_t yt,
                            int64_t lo, int64_t hi, int32_t rounding, int64_t *out)
{
    return requantize_one(v, M, zp_out, yt, lo, hi, rounding, out);
}

/* Thread count for the oracle's later parallel loops (n >= 1); timing
   only, the results do not depend on it. */
void oracle_set_threads(int n)
{
    if (n >= 1)
        omp_set_num_threads(n);
}

/* Number of OpenMP threads the oracle's parallel loops use. */
int oracle_threads(void)
{
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        n = omp_get_num_threads();
    }
    return n;
}
