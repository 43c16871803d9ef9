// Test infrastructure: drives the host side of libqnn (argument validation,
// the fixed-point multiplier, the kernel-choice file parser, error strings,
// NULL handling) with the address and undefined-behaviour sanitizers on the
// host code (tests/test_sanitizers.py builds it).  Needs no GPU: every call
// here fails validation, or reaches no device work, before any launch.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "qnn.h"

static int g_fail = 0;

static void expect(qnn_status got, qnn_status want, const char *what)
{
    if (got != want) {
        std::printf("%s: got %s, want %s (%s)\n", what, qnn_status_string(got), qnn_status_string(want),
                    qnn_last_error());
        g_fail = 1;
    }
}

int main(int argc, char **argv)
{
    int32_t m = 0, s = 0;
    const double Ms[] = {0.0, 1e-300, 2e-30, 1e-9, 0.25, 0.5, 1.0, 7.5, 1e8, 1.0737418e9};
    for (double M : Ms)
        (void)qnn_quantize_multiplier(M, &m, &s);
    expect(qnn_quantize_multiplier(-1.0, &m, &s), QNN_ERR_QPARAM, "negative multiplier");
    expect(qnn_quantize_multiplier(1.0, nullptr, &s), QNN_ERR_NULL, "null out");
    for (int c = 0; c <= 8; ++c)
        (void)std::strlen(qnn_status_string((qnn_status)c));
    (void)qnn_status_string((qnn_status)99);

    // conv validation: a valid description with one field broken at a time
    void *fake = (void *)0x10000;
    float xs = 0.02f, ws[64], ys = 0.05f;
    int32_t xz = 128, wz[64], yz = 0;
    for (int k = 0; k < 64; ++k)
        ws[k] = 0.01f, wz[k] = 0;
    qnn_qparams xq{&xs, &xz, 1}, wq{ws, wz, 1}, yq{&ys, &yz, 1};
    qnn_conv_params cp{1, 1, 1, 1, 1, 1, 1, 1};
    qnn_clamp act{INT32_MIN, INT32_MAX};
    auto conv = [&](qnn_dtype xt, int N, int H, int W, int C, int K, int R, int S, qnn_conv_params p, int ldc,
                    int coff, qnn_qparams w) {
        return qnn_conv2d(nullptr, fake, xt, N, H, W, C, xq, (const int8_t *)fake, K, R, S, w, nullptr, p, fake,
                          QNN_UINT8, yq, act, QNN_ROUND_HALF_UP, ldc, coff);
    };
    expect(conv(QNN_UINT8, 1, 8, 8, 16, 32, 3, 3, cp, 31, 0, wq), QNN_ERR_SHAPE, "y_ldc");
    expect(conv(QNN_UINT8, -1, 8, 8, 16, 32, 3, 3, cp, 32, 0, wq), QNN_ERR_SHAPE, "N");
    expect(conv(QNN_INT32, 1, 8, 8, 16, 32, 3, 3, cp, 32, 0, wq), QNN_ERR_DTYPE, "x dtype");
    {
        // x zero point 0 and w zero point 127: |x - zp| and |w - zp| reach 255
        int32_t z0 = 0, z127 = 127;
        const qnn_status st = qnn_conv2d(nullptr, fake, QNN_UINT8, 1, 1, 1, 33026, qnn_qparams{&xs, &z0, 1},
                                         (const int8_t *)fake, 4, 1, 1, qnn_qparams{ws, &z127, 1}, nullptr,
                                         qnn_conv_params{1, 1, 0, 0, 0, 0, 1, 1}, fake, QNN_UINT8, yq, act,
                                         QNN_ROUND_HALF_UP, 4, 0);
        expect(st, QNN_ERR_OVERFLOW, "overflow bound");
    }
    qnn_qparams wbad{ws, wz, 5};
    expect(conv(QNN_UINT8, 1, 8, 8, 16, 32, 3, 3, cp, 32, 0, wbad), QNN_ERR_QPARAM, "qparams length");
    expect(conv(QNN_UINT8, 1, 14000, 14000, 9, 4, 3, 3, cp, 4, 0, wq), QNN_ERR_UNSUPPORTED, "padded channels");
    expect(conv(QNN_UINT8, 1 << 20, 64, 64, 16, 32, 3, 3, cp, 32, 0, wq), QNN_ERR_UNSUPPORTED, "2^31 elements");
    expect(conv(QNN_UINT8, 0, 8, 8, 16, 32, 3, 3, cp, 32, 0, wq), QNN_OK, "empty batch");

    // uint8 weights: zero points outside [0, 255], and a dtype the calls do not take
    qnn_plan *p = nullptr;
    int32_t wz_bad[1] = {300};
    expect(qnn_conv2d_plan_create_wt(&p, nullptr, QNN_UINT8, 1, 8, 8, 16, xq, fake, QNN_UINT8, 32, 3, 3,
                                     qnn_qparams{ws, wz_bad, 1}, nullptr, cp, QNN_UINT8, yq, act,
                                     QNN_ROUND_HALF_UP, 32, 0),
           QNN_ERR_QPARAM, "uint8 weight zero point");
    expect(qnn_dense_plan_create_wt(&p, nullptr, QNN_UINT8, 4, 16, xq, fake, QNN_INT32, 8, wq, nullptr, QNN_INT8, yq,
                                    act, QNN_ROUND_HALF_UP, 8),
           QNN_ERR_DTYPE, "weight dtype");

    // requantize / add / pool validation
    expect(qnn_requantize(nullptr, fake, QNN_INT32, 16, 1, qnn_qparams{&xs, &xz, 1}, fake, QNN_UINT8, yq, act,
                          QNN_ROUND_HALF_UP),
           QNN_ERR_QPARAM, "int32 input zero point");
    expect(qnn_add(nullptr, nullptr, QNN_UINT8, xq, fake, QNN_UINT8, xq, 16, fake, QNN_UINT8, yq, act,
                   QNN_ROUND_HALF_UP),
           QNN_ERR_NULL, "add null");
    expect(qnn_pool2d(nullptr, fake, QNN_UINT8, 1, 4, 4, 8, 3, 3, qnn_conv_params{1, 1, 3, 0, 0, 0, 1, 1},
                      QNN_POOL_AVG, 0, 0, fake, QNN_ROUND_HALF_UP),
           QNN_ERR_SHAPE, "pool pad >= window");

    // plan handles
    expect(qnn_plan_run(nullptr, nullptr, fake, fake, nullptr), QNN_ERR_NULL, "run null plan");
    expect(qnn_plan_run_noalloc(nullptr, nullptr, fake, fake), QNN_ERR_NULL, "noalloc null plan");
    expect(qnn_plan_run_timed(nullptr, nullptr, fake, fake, nullptr, fake, fake), QNN_ERR_NULL, "timed null plan");
    (void)qnn_plan_workspace_size(nullptr);
    (void)qnn_plan_describe(nullptr);
    qnn_plan_destroy(nullptr);

    // the kernel-choice file parser: long, short and malformed lines
    if (argc > 1) {
        FILE *f = std::fopen(argv[1], "w");
        std::fprintf(f, "conv:x0:n1 2 3 1\nshort\n%0600d 1 2 3\n\n-- -1 -1 -1\nconv:y 2 3\n", 7);
        std::fclose(f);
        expect(qnn_set_tuning_file(argv[1]), QNN_OK, "tuning file");
        expect(qnn_set_tuning_file(nullptr), QNN_OK, "tuning file off");
    }
    std::printf("abi sanitizer run done\n");
    return g_fail;
}
