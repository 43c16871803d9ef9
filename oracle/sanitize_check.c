/*
 * Test infrastructure: a driver that runs every oracle entry point on small
 * seeded inputs (ragged shapes, strides, asymmetric padding, dilation,
 * depthwise, uint8 and int8 operands, all roundings, per-channel and
 * per-tensor parameters, int32 extremes, empty batches), built with the
 * address and undefined-behaviour sanitizers by tests/test_sanitizers.py.
 * It checks no values: the other oracle tests pin those.  Exit status 0
 * and no sanitizer report mean every access stayed inside its buffer and no
 * signed overflow or invalid shift occurred.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_quantize_multiplier(double M, int32_t *mult, int32_t *shift);
int64_t oracle_round_mul_shift(int64_t v, int32_t mult, int32_t shift, int rounding);
void oracle_conv_out_hw(const int32_t *shape, const int32_t *cp, int64_t *ho, int64_t *wo);
void oracle_conv2d_acc(const void *x, int32_t xt, int32_t zp_x, const void *w, int32_t wt, const int32_t *zp_w,
                       const int32_t *bias, const int32_t *shape, const int32_t *cp, int32_t depthwise,
                       int64_t *acc);
void oracle_conv2d_acc_points(const void *x, int32_t xt, int32_t zp_x, const void *w, int32_t wt,
                              const int32_t *zp_w, const int32_t *bias, const int32_t *shape, const int32_t *cp,
                              int32_t depthwise, const int64_t *idx, int64_t npts, int64_t *acc);
void oracle_dense_acc(const void *x, int32_t xt, int32_t zp_x, const void *w, int32_t wt, const int32_t *zp_w,
                      const int32_t *bias, int64_t M, int64_t Kd, int64_t Nd, int64_t *acc);
int oracle_requantize_acc(const int64_t *acc, int64_t Mrows, int64_t K, float s_x, const float *s_w, int32_t nw,
                          float s_y, int32_t zp_y, int32_t yt, int64_t lo, int64_t hi, int32_t rounding, void *y,
                          int64_t y_ldc, int64_t y_coff);
int oracle_requantize_points(const int64_t *acc, const int64_t *idx, int64_t npts, int64_t K, float s_x,
                             const float *s_w, int32_t nw, float s_y, int32_t zp_y, int32_t yt, int64_t lo,
                             int64_t hi, int32_t rounding, int64_t *out);
int oracle_requantize(const void *x, int32_t xt, int64_t count, int64_t channels, const float *s_in,
                      const int32_t *zp_in, int32_t n_in, const float *s_out, const int32_t *zp_out, int32_t n_out,
                      int32_t yt, int64_t lo, int64_t hi, int32_t rounding, void *y);
int oracle_add(const void *a, int32_t at, float s_a, int32_t zp_a, const void *b, int32_t bt, float s_b,
               int32_t zp_b, int64_t count, float s_o, int32_t zp_o, int32_t yt, int64_t lo, int64_t hi,
               int32_t rounding, void *y);
int oracle_pool2d(const void *x, int32_t xt, const int32_t *shape, const int32_t *pp, int32_t mode,
                  int32_t count_pad, int32_t zp, int32_t rounding, void *y);

static uint64_t g_state = 0x9E3779B97F4A7C15ull;

static uint32_t rnd(void)
{
    g_state ^= g_state << 13;
    g_state ^= g_state >> 7;
    g_state ^= g_state << 17;
    return (uint32_t)(g_state >> 16);
}

static int irange(int lo, int hi) { return lo + (int)(rnd() % (uint32_t)(hi - lo + 1)); }

/* exact-size heap buffers, so that the address sanitizer sees every overrun */
static void *buf(size_t bytes) { return malloc(bytes ? bytes : 1); }

static void fill8(void *p, size_t n)
{
    for (size_t i = 0; i < n; ++i)
        ((uint8_t *)p)[i] = (uint8_t)rnd();
}

static void conv_case(int depthwise, int xt, int wt)
{
    const int N = irange(0, 2), H = irange(1, 9), W = irange(1, 9), C = irange(1, 7);
    const int K = depthwise ? C : irange(1, 6);
    const int dh = irange(1, 2), dw = irange(1, 2);
    const int R = irange(1, 3), S = irange(1, 3);
    const int pt = irange(0, 2), pl = irange(0, 2), pb = irange(0, 2), pr = irange(0, 2);
    if ((R - 1) * dh + 1 > H + pt + pb || (S - 1) * dw + 1 > W + pl + pr)
        return;
    const int32_t shape[7] = {N, H, W, C, K, R, S};
    const int32_t cp[8] = {irange(1, 3), irange(1, 3), pt, pl, pb, pr, dh, dw};
    int64_t Ho, Wo;
    oracle_conv_out_hw(shape, cp, &Ho, &Wo);
    const size_t nx = (size_t)N * H * W * C, nw = depthwise ? (size_t)R * S * C : (size_t)K * R * S * C;
    void *x = buf(nx), *w = buf(nw);
    fill8(x, nx);
    fill8(w, nw);
    int32_t *zpw = buf(sizeof(int32_t) * K), *bias = buf(sizeof(int32_t) * K);
    for (int k = 0; k < K; ++k) {
        zpw[k] = wt == 0 ? irange(0, 255) : irange(-128, 127);
        bias[k] = irange(-100000, 100000);
    }
    const int64_t M = N * Ho * Wo;
    int64_t *acc = buf(sizeof(int64_t) * (size_t)(M * K));
    oracle_conv2d_acc(x, xt, xt == 0 ? irange(0, 255) : irange(-128, 127), w, wt, zpw, bias, shape, cp, depthwise,
                      acc);
    const int64_t np = M * K;
    int64_t *idx = buf(sizeof(int64_t) * (size_t)np), *pts = buf(sizeof(int64_t) * (size_t)np);
    for (int64_t i = 0; i < np; ++i)
        idx[i] = np - 1 - i;
    oracle_conv2d_acc_points(x, xt, 3, w, wt, zpw, NULL, shape, cp, depthwise, idx, np, pts);
    /* requantize of these accumulators, per channel, every rounding, slices */
    float sw[8];
    for (int k = 0; k < K; ++k)
        sw[k] = 0.001f * (float)irange(1, 9);
    for (int r = 0; r < 3; ++r) {
        const int yt = r == 2 ? 2 : r;   /* uint8, int8, int32 */
        const int64_t ldc = K + 3;
        void *y = buf((size_t)(M ? M : 1) * (size_t)ldc * (yt == 2 ? 4 : 1));
        oracle_requantize_acc(acc, M, K, 0.02f, sw, K, yt == 2 ? 1e-5f : 0.5f, yt == 2 ? 0 : 7, yt,
                              -2147483648ll, 2147483647ll, r, y, ldc, 2);
        int64_t *out = buf(sizeof(int64_t) * (size_t)np);
        oracle_requantize_points(pts, idx, np, K, 0.02f, sw, 1, 0.5f, -3, 1, -128, 127, r, out);
        free(out);
        free(y);
    }
    free(x), free(w), free(zpw), free(bias), free(acc), free(idx), free(pts);
}

int main(void)
{
    int32_t m, s;
    const double Ms[] = {1e-300, 2e-30, 1e-9, 0.001, 0.5, 0.999999, 1.0, 3.0, 1e8, 1e9};
    for (size_t i = 0; i < sizeof Ms / sizeof Ms[0]; ++i)
        if (oracle_quantize_multiplier(Ms[i], &m, &s) == 0)
            for (int r = 0; r < 3; ++r) {
                (void)oracle_round_mul_shift(2147483647ll, m, s, r);
                (void)oracle_round_mul_shift(-2147483648ll, m, s, r);
                (void)oracle_round_mul_shift(0, m, s, r);
            }
    for (int t = 0; t < 400; ++t)
        conv_case(t % 3 == 0, t % 2, (t / 2) % 2);
    /* dense, uint8 and int8 operands */
    for (int t = 0; t < 50; ++t) {
        const int M = irange(0, 5), Kd = irange(1, 40), Nd = irange(1, 9);
        void *x = buf((size_t)M * Kd), *w = buf((size_t)Nd * Kd);
        fill8(x, (size_t)M * Kd);
        fill8(w, (size_t)Nd * Kd);
        int32_t *zpw = buf(sizeof(int32_t) * Nd);
        for (int j = 0; j < Nd; ++j)
            zpw[j] = irange(-20, 20);
        int64_t *acc = buf(sizeof(int64_t) * (size_t)M * Nd);
        oracle_dense_acc(x, t % 2, 5, w, (t / 2) % 2, zpw, NULL, M, Kd, Nd, acc);
        free(x), free(w), free(zpw), free(acc);
    }
    /* standalone requantize and add over every dtype pair and rounding */
    for (int xt = 0; xt < 3; ++xt)
        for (int yt = 0; yt < 3; ++yt)
            for (int r = 0; r < 3; ++r) {
                const int64_t count = irange(0, 300), ch = 6;
                const size_t es = xt == 2 ? 4 : 1, ys = yt == 2 ? 4 : 1;
                void *x = buf((size_t)count * es), *y = buf((size_t)count * ys);
                fill8(x, (size_t)count * es);
                const float si[6] = {0.1f, 0.2f, 0.3f, 0.4f, 0.5f, 0.6f}, so[1] = {0.05f};
                const int32_t zi[6] = {0}, zo[1] = {0};
                oracle_requantize(x, xt, count, ch, si, zi, 6, so, zo, 1, yt, -2147483648ll, 2147483647ll, r, y);
                if (xt < 2 && yt < 2)
                    oracle_add(x, xt, 0.1f, 3, x, xt, 0.3f, -2, count, 0.2f, 1, yt, -128, 255, r, y);
                free(x), free(y);
            }
    /* pooling: average (both padding modes, both roundings) and max */
    for (int t = 0; t < 100; ++t) {
        const int N = irange(0, 2), H = irange(1, 8), W = irange(1, 8), C = irange(1, 5);
        const int R = irange(1, 4), S = irange(1, 4);
        const int32_t pp[6] = {irange(1, 3), irange(1, 3), irange(0, R - 1), irange(0, S - 1), irange(0, R - 1),
                               irange(0, S - 1)};
        if (R > H + pp[2] + pp[4] || S > W + pp[3] + pp[5])
            continue;
        const int32_t shape[6] = {N, H, W, C, R, S};
        const int64_t Ho = (H + pp[2] + pp[4] - R) / pp[0] + 1, Wo = (W + pp[3] + pp[5] - S) / pp[1] + 1;
        void *x = buf((size_t)N * H * W * C), *y = buf((size_t)N * Ho * Wo * C);
        fill8(x, (size_t)N * H * W * C);
        (void)oracle_pool2d(x, t % 2, shape, pp, t % 3 == 0, (t / 3) % 2, t % 2 ? -4 : 9, (t / 6) % 2, y);
        free(x), free(y);
    }
    printf("oracle sanitizer run done\n");
    return 0;
}
