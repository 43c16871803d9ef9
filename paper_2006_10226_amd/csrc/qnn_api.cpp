// C ABI of libqnn: argument validation, plan creation (per-channel
// fixed-point multipliers, folded constants, packed weights), kernel choice
// and launches.  See include/qnn.h for the contract of every entry point.
#include "qnn.h"
#include "qnn_internal.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cerrno>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

using namespace qnn;

qnn::LaunchEvents &qnn::launch_events()
{
    static thread_local LaunchEvents ev;
    return ev;
}

namespace {

thread_local std::string g_last_error;

qnn_status fail(qnn_status s, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}

qnn_status hip_fail(hipError_t e, const char *what)
{
    return fail(QNN_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr)                                 \
    do {                                              \
        hipError_t e_ = (expr);                       \
        if (e_ != hipSuccess)                         \
            return hip_fail(e_, #expr);               \
    } while (0)

struct Range {
    int64_t lo, hi;
};

bool dtype_range(qnn_dtype t, Range *r)
{
    switch (t) {
    case QNN_UINT8: *r = {0, 255}; return true;
    case QNN_INT8: *r = {-128, 127}; return true;
    case QNN_INT32: *r = {INT32_MIN, INT32_MAX}; return true;
    default: return false;
    }
}

const char *dtype_name(qnn_dtype t)
{
    switch (t) {
    case QNN_UINT8: return "uint8";
    case QNN_INT8: return "int8";
    case QNN_INT32: return "int32";
    default: return "?";
    }
}

// Fixed-point multiplier of Sec. III-B (the library's own derivation; see
// qnn_quantize_multiplier in qnn.h for the rule).
bool derive_multiplier(double M, int32_t *mult, int32_t *shift)
{
    if (!(M >= 0.0) || !std::isfinite(M))
        return false;
    if (M == 0.0) {
        *mult = 0;
        *shift = 1;
        return true;
    }
    int e;
    const double f = std::frexp(M, &e);
    int64_t q = (int64_t)std::floor(std::ldexp(f, 31) + 0.5);
    if (q == (int64_t(1) << 31)) {
        q >>= 1;
        ++e;
    }
    const int n = 31 - e;
    if (n < 1)
        return false;
    *mult = (int32_t)q;
    *shift = n;
    return true;
}

qnn_status check_qparams(const qnn_qparams &q, const char *what, int32_t n_allowed, qnn_dtype zp_dtype,
                         bool allow_zero_scale)
{
    if (!q.scale || !q.zero_point)
        return fail(QNN_ERR_NULL, "%s: scale / zero_point array is NULL", what);
    if (q.n != 1 && q.n != n_allowed)
        return fail(QNN_ERR_QPARAM, "%s: qparams length %d, expected 1 or %d", what, q.n, n_allowed);
    Range r;
    dtype_range(zp_dtype, &r);
    for (int i = 0; i < q.n; ++i) {
        const float s = q.scale[i];
        if (!std::isfinite(s) || s < 0.0f || (s == 0.0f && !allow_zero_scale))
            return fail(QNN_ERR_QPARAM, "%s: scale[%d] = %g is not a finite positive value", what, i, (double)s);
        if (q.zero_point[i] < r.lo || q.zero_point[i] > r.hi)
            return fail(QNN_ERR_QPARAM, "%s: zero_point[%d] = %d outside the %s range", what, i, q.zero_point[i],
                        dtype_name(zp_dtype));
    }
    return QNN_OK;
}

// Output clamp intersected with the output dtype range.
qnn_status out_bounds(qnn_dtype yt, qnn_clamp act, int32_t *lo, int32_t *hi)
{
    Range r;
    if (!dtype_range(yt, &r))
        return fail(QNN_ERR_DTYPE, "unknown output dtype %d", (int)yt);
    const int64_t l = std::max<int64_t>(r.lo, act.lo), h = std::min<int64_t>(r.hi, act.hi);
    if (l > h)
        return fail(QNN_ERR_QPARAM, "empty output clamp [%d, %d] for %s", act.lo, act.hi, dtype_name(yt));
    *lo = (int32_t)l;
    *hi = (int32_t)h;
    return QNN_OK;
}

int env_int(const char *name, int dflt)
{
    const char *v = std::getenv(name);
    return v && *v ? std::atoi(v) : dflt;
}

enum PlanKind { PLAN_CONV = 0, PLAN_DW = 1, PLAN_REQ = 2 };

}  // namespace

// One implicit-GEMM kernel configuration: family and tile enum value.
enum KernelFamily { FAM_GATHER = 0, FAM_TAP = 1, FAM_DMA = 2, FAM_WAVE = 3, FAM_HALO = 4, FAM_WIN = 5 };
struct ConvKernel {
    int fam = FAM_GATHER;
    int tile = TILE_64x64;
    int split = 1;   // LDS-direct ring kernel: K-step parts per tile
};

struct qnn_plan {
    PlanKind kind;
    // conv / dense
    ConvArgs conv{};
    int avec = 16, mode = OUT_REQUANT;
    ConvKernel ker;             // kernel family and tile that run_plan launches
    bool term3 = false;
    // the conv output's own quantization (the first input of a fused
    // residual add), and whether an add is fused (qnn_plan_set_residual)
    float y_scale = 1.0f;
    int32_t y_zp = 0;
    int y_dt = QNN_UINT8;
    bool fused = false;
    int32_t *addtab = nullptr;  // the fused add's term tables (AddArgs::tab), plan-owned
    size_t ws_asum_bytes = 0, ws_xpad_bytes = 0;
    size_t ws_cnt_bytes = 0, ws_part_bytes = 0;   // split reduction: counters, partial sums
    int32_t C_in = 0;           // channels of the caller's x (before padding to a.C)
    bool rowpack = false;       // row-pair mode: x is copied into a zero-point padded image
    int32_t H_in = 0, W_in = 0, pt_in = 0, pl_in = 0;   // caller's image and pads (row-pair mode)
    uint8_t pad_zp = 0;         // zero point byte written into padded channels
    // depthwise
    DwArgs dw{};
    bool dw3 = false;               // the 3x3 dot-product kernel applies
    const ChanRec *chan3 = nullptr; // its channel records (constant with the zero-point terms)
    // requantize
    ReqArgs req{};
    int xdt = 0, ydt = 0;
    // memory
    void *dev = nullptr;      // packed weights + tables
    void *ws_own = nullptr;   // plan-owned workspace
    size_t ws_bytes = 0;
    std::string desc;
};

namespace {

void free_plan(qnn_plan *p)
{
    if (!p)
        return;
    if (p->dev)
        (void)hipFree(p->dev);
    if (p->ws_own)
        (void)hipFree(p->ws_own);
    if (p->addtab)
        (void)hipFree(p->addtab);
    delete p;
}

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct ConvDesc {
    qnn_dtype xt;
    int32_t N, H, W, C;
    qnn_qparams xq;
    const int8_t *w;
    int32_t K, R, S;
    qnn_qparams wq;
    const int32_t *bias;
    qnn_conv_params cp;
    qnn_dtype yt;
    qnn_qparams yq;
    qnn_clamp act;
    qnn_rounding rnd;
    int32_t y_ldc, y_coff;
    bool depthwise;
};

// Shared validation of conv / depthwise / dense descriptors.  Fills the
// output size, output clamp and per-channel multipliers.
qnn_status validate_conv(const ConvDesc &d, int32_t *Ho, int32_t *Wo, int32_t *lo, int32_t *hi,
                         std::vector<int32_t> *mult, std::vector<int32_t> *shift)
{
    const char *op = d.depthwise ? "depthwise_conv2d" : "conv2d";
    if (d.xt != QNN_UINT8 && d.xt != QNN_INT8)
        return fail(QNN_ERR_DTYPE, "%s: input dtype must be uint8 or int8", op);
    if (d.yt != QNN_UINT8 && d.yt != QNN_INT8 && d.yt != QNN_INT32)
        return fail(QNN_ERR_DTYPE, "%s: output dtype must be uint8, int8 or int32", op);
    if (d.rnd < QNN_ROUND_HALF_UP || d.rnd > QNN_ROUND_TWO_STAGE)
        return fail(QNN_ERR_QPARAM, "%s: unknown rounding %d", op, (int)d.rnd);
    if (d.N < 0 || d.H < 1 || d.W < 1 || d.C < 1 || d.K < 1 || d.R < 1 || d.S < 1)
        return fail(QNN_ERR_SHAPE, "%s: sizes must be positive (N >= 0)", op);
    const qnn_conv_params &c = d.cp;
    if (c.stride_h < 1 || c.stride_w < 1 || c.dil_h < 1 || c.dil_w < 1 || c.pad_top < 0 || c.pad_left < 0 ||
        c.pad_bottom < 0 || c.pad_right < 0)
        return fail(QNN_ERR_SHAPE, "%s: strides/dilations must be >= 1 and pads >= 0", op);
    const int64_t hn = (int64_t)d.H + c.pad_top + c.pad_bottom - (int64_t)c.dil_h * (d.R - 1) - 1;
    const int64_t wn = (int64_t)d.W + c.pad_left + c.pad_right - (int64_t)c.dil_w * (d.S - 1) - 1;
    if (hn < 0 || wn < 0)
        return fail(QNN_ERR_SHAPE, "%s: filter larger than the padded input", op);
    *Ho = (int32_t)(hn / c.stride_h + 1);
    *Wo = (int32_t)(wn / c.stride_w + 1);
    if (d.y_coff < 0 || (int64_t)d.y_ldc < (int64_t)d.y_coff + d.K)
        return fail(QNN_ERR_SHAPE, "%s: need y_coff >= 0 and y_ldc >= y_coff + %d (got %d, %d)", op, d.K,
                    d.y_ldc, d.y_coff);
    const int64_t xelems = (int64_t)d.N * d.H * d.W * d.C;
    const int64_t M = (int64_t)d.N * *Ho * *Wo;
    if (xelems >= (int64_t(1) << 31) || M * d.y_ldc >= (int64_t(1) << 31) ||
        (int64_t)d.R * d.S * d.C >= (int64_t(1) << 24))
        return fail(QNN_ERR_UNSUPPORTED, "%s: tensors of 2^31 or more elements are not supported", op);
    if (!d.w)
        return fail(QNN_ERR_NULL, "%s: weight pointer is NULL", op);

    qnn_status s;
    if ((s = check_qparams(d.xq, "x qparams", 1, d.xt, false)) != QNN_OK)
        return s;
    if ((s = check_qparams(d.wq, "w qparams", d.K, QNN_INT8, true)) != QNN_OK)
        return s;
    *lo = INT32_MIN;
    *hi = INT32_MAX;
    mult->assign(d.K, 0);
    shift->assign(d.K, 1);
    if (d.yt != QNN_INT32) {
        if ((s = check_qparams(d.yq, "y qparams", 1, d.yt, false)) != QNN_OK)
            return s;
        if ((s = out_bounds(d.yt, d.act, lo, hi)) != QNN_OK)
            return s;
        for (int k = 0; k < d.K; ++k) {
            const double sw = (double)d.wq.scale[d.wq.n == 1 ? 0 : k];
            const double Mk = ((double)d.xq.scale[0] * sw) / (double)d.yq.scale[0];
            int32_t m, n;
            if (!derive_multiplier(Mk, &m, &n))
                return fail(QNN_ERR_QPARAM, "%s: requantize multiplier %g of channel %d is out of range", op, Mk, k);
            (*mult)[k] = m;
            (*shift)[k] = n > 63 ? 63 : n;
        }
    }
    return QNN_OK;
}

// Accumulator bound (host copy of the bias): J * max|x - zp_x| * max|w - zp_w| + |bias| < 2^31.
qnn_status check_overflow(const ConvDesc &d, int64_t J, const std::vector<int32_t> &bias_h)
{
    Range xr;
    dtype_range(d.xt, &xr);
    const int64_t zx = d.xq.zero_point[0];
    const int64_t ax = std::max(zx - xr.lo, xr.hi - zx);
    for (int k = 0; k < d.K; ++k) {
        const int64_t zw = d.wq.zero_point[d.wq.n == 1 ? 0 : k];
        const int64_t aw = std::max(zw + 128, 127 - zw);
        const int64_t b = bias_h.empty() ? 0 : std::llabs((long long)bias_h[k]);
        if (J * ax * aw + b >= (int64_t(1) << 31))
            return fail(QNN_ERR_OVERFLOW,
                        "accumulator bound J*|x-zp|*|w-zp|+|bias| = %lld for channel %d does not fit int32",
                        (long long)(J * ax * aw + b), k);
    }
    return QNN_OK;
}

qnn_status read_bias(const int32_t *bias, int n, hipStream_t st, std::vector<int32_t> *out)
{
    out->clear();
    if (!bias)
        return QNN_OK;
    out->resize(n);
    HIP_TRY(hipMemcpyAsync(out->data(), bias, sizeof(int32_t) * n, hipMemcpyDeviceToHost, st));
    HIP_TRY(hipStreamSynchronize(st));
    return QNN_OK;
}

TileShape kernel_shape(const ConvKernel &k)
{
    switch (k.fam) {
    case FAM_WAVE: return {64, 64, 64};
    case FAM_HALO: return {64, 64, 64};
    case FAM_WIN: return {win_channels(k.tile), 64, 64};
    case FAM_DMA: return dma_tile_shape(k.tile);
    case FAM_TAP: return tap_tile_shape(k.tile);
    default: return tile_shape(k.tile);
    }
}

int device_cus();

// Candidate kernels for a conv of M pixels x K channels with C4 channels
// per tap and reduction J.  QNN_DMA / QNN_TAP / QNN_TILE=<n> force one
// configuration when it is eligible (for sweeps and tests).  one_tap: a
// 1x1 filter, whose K-steps may end past the pixel's channels (C4 % 16 ==
// 0): the extra bytes are the next pixels' and meet zero weights.
std::vector<ConvKernel> conv_candidates(int64_t M, int K, int C4, int J, bool tap_ok, bool dma_ok, bool one_tap)
{
    (void)M;
    (void)K;
    std::vector<ConvKernel> c;
    const int f_dma = env_int("QNN_DMA", -1), f_tap = env_int("QNN_TAP", -1), f_tile = env_int("QNN_TILE", -1);
    const int f_wave = env_int("QNN_WAVE", -1);
    // the wave kernel starts its split reduction at tap (ks / (C / 64)):
    // whole 64-channel steps only
    const bool wave_ok = dma_ok && C4 % 64 == 0;
    auto tap_fits = [&](int t) { return C4 % tap_tile_shape(t).bk == 0 || one_tap; };
    if ((f_wave == 1 || f_wave == 2 || f_wave == 4 || f_wave == 8) && wave_ok)
        return {{FAM_WAVE, f_wave}};
    if (f_dma >= 0 && f_dma < DMA_COUNT && dma_ok && (!dma_short(f_dma) || (J + 63) / 64 <= dma_stages(f_dma))) {
        // QNN_KSPLIT=<parts> with a forced ring configuration that has a split form
        const int f_split = env_int("QNN_KSPLIT", 1);
        if (f_split > 1 && dma_splits(f_dma) && C4 % 64 == 0 && J / 64 >= f_split)
            return {{FAM_DMA, f_dma, f_split}};
        return {{FAM_DMA, f_dma}};
    }
    if (f_tap >= 0 && f_tap < TAP_COUNT && tap_ok && tap_fits(f_tap))
        return {{FAM_TAP, f_tap}};
    if (f_tile >= 0 && f_tile < TILE_COUNT)
        return {{FAM_GATHER, f_tile}};
    if (wave_ok && env_int("QNN_WAVE", -1) != -2)
        for (int sp : {1, 2, 4, 8})
            if (sp == 1 || J / 64 >= 2 * sp)
                c.push_back({FAM_WAVE, sp});
    if (tap_ok && env_int("QNN_TAP", -1) != -2)
        for (int t = 0; t < TAP_COUNT; ++t)
            if (tap_fits(t))
                c.push_back({FAM_TAP, t});
    if (dma_ok && env_int("QNN_DMA", -1) != -2) {
        for (int t : {DMA_128x128_S4, DMA_128x64_S4, DMA_64x128_S4, DMA_64x64_S4, DMA_256x128_S4, DMA_128x256_S4,
                      DMA_128x128_S8, DMA_128x64_S8, DMA_64x64_S8, DMA_64x128_S8, DMA_64x64_S16})
            c.push_back({FAM_DMA, t});
        // two K-step groups per tile: reductions of at least 8 steps
        if ((J + 63) / 64 >= 8)
            for (int t : {DMA_128x64_K2, DMA_64x64_K2, DMA_128x128_K2})
                c.push_back({FAM_DMA, t});
        // short reductions: every K-step in flight at once
        for (int t = DMA_64x128_R1; t < DMA_COUNT; ++t)
            if (dma_short(t) && (J + 63) / 64 <= dma_stages(t))
                c.push_back({FAM_DMA, t});
        // split reductions, for grids of fewer tiles than about two per CU:
        // each tile's K-steps in parts of at least three steps, run by
        // separate workgroups whose partial sums the last one adds
        if (C4 % 64 == 0 && env_int("QNN_SPLIT", 1) != 0) {
            const int nk = J / 64;
            const int64_t cus = device_cus();
            for (int t = 0; t < DMA_COUNT; ++t) {
                if (!dma_splits(t))
                    continue;
                const TileShape ts = dma_tile_shape(t);
                const int64_t tiles = (int64_t)((K + ts.tc - 1) / ts.tc) * ((M + ts.tp - 1) / ts.tp);
                if (tiles >= 2 * cus)
                    continue;
                for (int sp : {2, 3, 4, 6, 8, 12, 16})
                    if (nk >= 3 * sp && tiles * sp <= 4 * cus)
                        c.push_back({FAM_DMA, t, sp});
            }
        }
    }
    if (c.empty() || C4 % 64 != 0) {
        // the general gather kernel (short reductions use the 64-deep
        // K-step); for 1x1 filters with partial K-steps it competes with
        // the tap-walk kernels, which read up to 48 bytes past each pixel
        const size_t first = c.size();
        c.push_back({FAM_GATHER, J <= 64 ? TILE_64x64_K64 : TILE_64x64});
        for (int t : {TILE_64x64_K64, TILE_64x128, TILE_128x64, TILE_128x128})
            if (t != c[first].tile)
                c.push_back({FAM_GATHER, t});
    }
    return c;
}

// Tiling of the launched kernel: tile counts, K-steps, persistent grid.
// The padding correction tables (pcorr_tab, pcls_tab) belong to the
// LDS-direct kernel only: the other families gather zp_x themselves.
void set_tiling(ConvArgs &a, const ConvKernel &k, int avec, const int32_t *pcorr_tab, const uint8_t *pcls_tab)
{
    const TileShape ts = kernel_shape(k);
    const bool zero_pad = k.fam == FAM_DMA || k.fam == FAM_WAVE;   // gathers read x = 0 outside the image
    a.pcorr = zero_pad ? pcorr_tab : nullptr;
    a.pcls = zero_pad ? pcls_tab : nullptr;
    const int64_t tiles_c = (a.K + ts.tc - 1) / ts.tc;
    int64_t ntiles = tiles_c * (((int64_t)a.M + ts.tp - 1) / ts.tp);
    if (k.fam == FAM_HALO) {
        // one wave tile is whole output rows of one image
        const long long tp = halo_pixel_tiles(a);
        ntiles = tp < 0 ? -1 : tiles_c * tp;
    } else if (k.fam == FAM_WIN) {
        const long long wg = win_workgroups_per_ctile(a, k.tile);
        ntiles = wg < 0 ? -1 : tiles_c * wg;
    }
    a.tiles_c = (int)tiles_c;
    a.ntiles = ntiles >= 0 && ntiles < (int64_t(1) << 31) - 8 ? (int)ntiles : -1;
    a.nk = (a.J + ts.bk - 1) / ts.bk;
    a.ksplit = k.fam == FAM_DMA ? k.split : 1;
    a.nblocks = 0;
    if (k.fam == FAM_GATHER && a.ntiles >= 0) {
        // persistent grid: as many workgroups as stay resident, a multiple
        // of 8 (one share per XCD), never more than there are tiles
        const size_t dyn = a.chan_in_lds ? (size_t)a.Kpad * sizeof(ChanRec) : 0;
        const int64_t resident = (int64_t)device_cus() * conv_blocks_per_cu(k.tile, avec, dyn);
        a.nblocks = (int)std::min<int64_t>((ntiles + 7) / 8 * 8, std::max<int64_t>(8, resident / 8 * 8));
    }
}

hipError_t launch_conv_kernel(const ConvArgs &a, const ConvKernel &k, int avec, hipStream_t st)
{
    switch (k.fam) {
    case FAM_WAVE: return launch_conv_wave(a, k.tile, st);
    case FAM_HALO: return launch_conv_halo(a, k.tile, st);
    case FAM_WIN: return launch_conv_window(a, k.tile, st);
    case FAM_DMA: return launch_conv_dma(a, k.tile, st);
    case FAM_TAP: return launch_conv_tap(a, k.tile, st);
    default: return launch_conv(a, k.tile, avec, st);
    }
}

// Times every candidate on the plan's shape and returns the fastest.
// Scratch activations (a constant fill), output and window sums are
// allocated for the measurement and freed again.
qnn_status autotune_conv(const ConvArgs &base, const std::vector<ConvKernel> &cands, int avec, bool term3,
                         const int32_t *pcorr_tab, const uint8_t *pcls_tab, hipStream_t st, ConvKernel *best)
{
    const size_t xb = align_up((size_t)base.N * base.H * base.W * base.C, 256);
    const size_t elem = base.mode == OUT_INT32 ? 4 : 1;
    const size_t yb = align_up((size_t)base.M * base.y_ldc * elem, 256);
    const size_t sb = align_up((size_t)base.M * sizeof(int32_t), 256);
    // split reductions: counters (zeroed, reset by every launch) and partial sums
    size_t cb = 0, pb = 0;
    for (const ConvKernel &k : cands) {
        if (k.fam != FAM_DMA || k.split <= 1)
            continue;
        const TileShape ts = kernel_shape(k);
        const size_t tiles = (size_t)((base.K + ts.tc - 1) / ts.tc) * ((base.M + ts.tp - 1) / ts.tp);
        cb = std::max(cb, align_up(tiles * sizeof(int32_t), 256));
        pb = std::max(pb, tiles * k.split * ts.tc * ts.tp * sizeof(int32_t));
    }
    void *buf = nullptr;
    hipError_t e = hipMalloc(&buf, xb + yb + sb + cb + pb);
    if (e != hipSuccess)
        return fail(QNN_ERR_ALLOC, "hipMalloc of %zu bytes for kernel tuning failed", xb + yb + sb + cb + pb);
    // Each timed launch starts with cold caches, as a layer does inside a
    // network: a pass over more than the L2s and the 256 MB last-level cache
    // runs before it.  (Without the buffer the timing is warm.)
    const size_t flush_bytes = size_t(320) << 20;
    void *flush = nullptr;
    if (hipMalloc(&flush, flush_bytes) != hipSuccess)
        flush = nullptr;
    // The eviction reads the whole buffer through the caches, then writes 16
    // MB of it: the caches then hold clean lines plus some dirty ones, as a
    // layer inside the stack finds them after its predecessor's output.
    // QNN_TUNE_FLUSH=0 fills the whole buffer instead (all lines dirty).
    const bool sweep = env_int("QNN_TUNE_FLUSH", 1) != 0;
    auto evict = [&](int r) -> hipError_t {
        if (!sweep)
            return hipMemsetAsync(flush, r, flush_bytes, st);
        hipError_t er = launch_cache_sweep(flush, flush_bytes, (int *)buf, st);
        return er != hipSuccess ? er : hipMemsetAsync(flush, r, size_t(16) << 20, st);
    };
    hipEvent_t e0 = nullptr, e1 = nullptr;
    qnn_status s = QNN_OK;
    float best_ms = 1e30f;
    ConvArgs a = base;
    a.x = (const uint8_t *)buf;
    a.y = (char *)buf + xb;
    a.asum = term3 ? (const int32_t *)((char *)buf + xb + yb) : nullptr;
    a.cnt = cb ? (int32_t *)((char *)buf + xb + yb + sb) : nullptr;
    a.part = cb ? (int32_t *)((char *)buf + xb + yb + sb + cb) : nullptr;
    if ((e = hipMemsetAsync(buf, 0x35, xb + yb + sb, st)) != hipSuccess ||
        (cb && (e = hipMemsetAsync((char *)buf + xb + yb + sb, 0, cb, st)) != hipSuccess) ||
        (e = hipEventCreate(&e0)) != hipSuccess ||
        (e = hipEventCreate(&e1)) != hipSuccess) {
        s = hip_fail(e, "kernel tuning set-up");
    } else {
        for (const ConvKernel &k : cands) {
            set_tiling(a, k, avec, pcorr_tab, pcls_tab);
            if (a.ntiles < 0)
                continue;
            float t = 0;
            // one untimed launch, then the median of five cold launches
            if ((e = launch_conv_kernel(a, k, avec, st)) != hipSuccess)
                break;
            constexpr int kRuns = 5;
            float runs[kRuns];
            for (int r = 0; r < kRuns && e == hipSuccess; ++r) {
                if (flush && (e = evict(r)) != hipSuccess)
                    break;
                if ((e = hipEventRecord(e0, st)) != hipSuccess || (e = launch_conv_kernel(a, k, avec, st)) != hipSuccess ||
                    (e = hipEventRecord(e1, st)) != hipSuccess || (e = hipEventSynchronize(e1)) != hipSuccess ||
                    (e = hipEventElapsedTime(&runs[r], e0, e1)) != hipSuccess)
                    break;
            }
            if (e != hipSuccess)
                break;
            std::sort(runs, runs + kRuns);
            t = runs[kRuns / 2];
            if (t < best_ms) {
                best_ms = t;
                *best = k;
            }
        }
        if (e != hipSuccess)
            s = hip_fail(e, "kernel tuning");
    }
    if (e0)
        (void)hipEventDestroy(e0);
    if (e1)
        (void)hipEventDestroy(e1);
    (void)hipStreamSynchronize(st);
    (void)hipFree(buf);
    if (flush)
        (void)hipFree(flush);
    return s;
}

// Kernel choices kept in a text file (qnn_set_tuning_file): one line per
// timed shape, "<key> <family> <config>".  A plan whose key is listed takes
// that choice without timing, provided it is still among its candidates.
std::mutex g_tune_mu;
std::string g_tune_path;
std::map<std::string, ConvKernel> g_tune;

std::string tune_key(const ConvDesc &d, bool term3, size_t ncls, bool fast)
{
    char buf[256];
    snprintf(buf, sizeof buf, "conv:x%d:n%d:h%d:w%d:c%d:k%d:r%d:s%d:st%dx%d:p%d,%d,%d,%d:d%dx%d:y%d:t%d:b%zu:f%d:l%d,%d",
             (int)d.xt, d.N, d.H, d.W, d.C, d.K, d.R, d.S, d.cp.stride_h, d.cp.stride_w, d.cp.pad_top,
             d.cp.pad_bottom, d.cp.pad_left, d.cp.pad_right, d.cp.dil_h, d.cp.dil_w, (int)d.yt, (int)term3, ncls,
             (int)fast, d.y_ldc, d.y_coff);
    return buf;
}

bool tune_lookup(const std::string &key, const std::vector<ConvKernel> &cands, ConvKernel *out)
{
    std::lock_guard<std::mutex> g(g_tune_mu);
    auto it = g_tune.find(key);
    if (it == g_tune.end())
        return false;
    for (const ConvKernel &k : cands)
        if (k.fam == it->second.fam && k.tile == it->second.tile && k.split == it->second.split) {
            *out = k;
            return true;
        }
    return false;
}

void tune_record(const std::string &key, const ConvKernel &k)
{
    std::lock_guard<std::mutex> g(g_tune_mu);
    g_tune[key] = k;
    if (g_tune_path.empty())
        return;
    if (FILE *f = std::fopen(g_tune_path.c_str(), "a")) {
        std::fprintf(f, "%s %d %d %d\n", key.c_str(), k.fam, k.tile, k.split);
        std::fclose(f);
    }
}

// Magic pair for n / d with 0 <= n < 2^31: with l = ceil(log2 d) and
// mul = ceil(2^(31+l) / d) < 2^32, n * mul / 2^(31+l) exceeds n / d by less
// than 2^-l <= 1/d, which never reaches the next integer, so
// n / d = umulhi(n, mul) >> (l - 1).  d == 1 is flagged by mul == 0.
void make_divider(uint32_t d, uint32_t &mul, uint32_t &shift)
{
    if (d <= 1) {
        mul = 0;
        shift = 0;
        return;
    }
    int l = 0;
    while ((1ull << l) < d)
        ++l;
    mul = (uint32_t)(((1ull << (31 + l)) + d - 1) / d);
    shift = (uint32_t)(l - 1);
}

// Border classes of the output pixels: the set of filter taps that fall
// outside the image depends on the output row through a row mask (valid
// r) and on the column through a column mask (valid s).  Each distinct
// (row mask, column mask) pair with an outside tap is a class; pixels with
// every tap inside get 255.
struct BorderClasses {
    std::vector<uint8_t> pcls;           // [M]
    std::vector<uint32_t> rmask, cmask;  // per class
    bool any = false;
};

bool border_classes(const ConvDesc &d, int Ho, int Wo, int64_t M, BorderClasses &bc)
{
    const uint32_t full_r = (1u << d.R) - 1, full_c = (1u << d.S) - 1;
    std::vector<uint32_t> ru, cu;
    std::vector<int> rcls(Ho), ccls(Wo);
    for (int oh = 0; oh < Ho; ++oh) {
        uint32_t m = 0;
        for (int r = 0; r < d.R; ++r) {
            const int64_t ih = (int64_t)oh * d.cp.stride_h - d.cp.pad_top + (int64_t)r * d.cp.dil_h;
            m |= (uint32_t)(ih >= 0 && ih < d.H) << r;
        }
        const auto it = std::find(ru.begin(), ru.end(), m);
        rcls[oh] = (int)(it - ru.begin());
        if (it == ru.end())
            ru.push_back(m);
    }
    for (int ow = 0; ow < Wo; ++ow) {
        uint32_t m = 0;
        for (int s = 0; s < d.S; ++s) {
            const int64_t iw = (int64_t)ow * d.cp.stride_w - d.cp.pad_left + (int64_t)s * d.cp.dil_w;
            m |= (uint32_t)(iw >= 0 && iw < d.W) << s;
        }
        const auto it = std::find(cu.begin(), cu.end(), m);
        ccls[ow] = (int)(it - cu.begin());
        if (it == cu.end())
            cu.push_back(m);
    }
    const size_t ncls = ru.size() * cu.size();
    if (ncls > 255)
        return false;
    bc.rmask.resize(ncls);
    bc.cmask.resize(ncls);
    std::vector<uint8_t> id(ncls);
    for (size_t rc = 0; rc < ru.size(); ++rc)
        for (size_t cc = 0; cc < cu.size(); ++cc) {
            const size_t c = rc * cu.size() + cc;
            bc.rmask[c] = ru[rc];
            bc.cmask[c] = cu[cc];
            const bool interior = ru[rc] == full_r && cu[cc] == full_c;
            id[c] = interior ? 255 : (uint8_t)c;
            bc.any |= !interior;
        }
    bc.pcls.resize((size_t)M);
    size_t m = 0;
    for (int n = 0; n < d.N; ++n)
        for (int oh = 0; oh < Ho; ++oh)
            for (int ow = 0; ow < Wo; ++ow)
                bc.pcls[m++] = id[(size_t)rcls[oh] * cu.size() + ccls[ow]];
    return true;
}

// LDS bytes one workgroup may use on the current device.
int device_lds_per_block()
{
    static int bytes = 0;
    if (!bytes) {
        int dev = 0, n = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&n, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess && n > 0)
            bytes = n;
        else
            bytes = 64 * 1024;
    }
    return bytes;
}

int device_cus()
{
    static int cus = 0;
    if (!cus) {
        int dev = 0, n = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
            cus = n;
        else
            cus = 256;
    }
    return cus;
}

// tune: time the candidate kernels when the kernel-choice records hold no
// choice for this shape (plans); one-shot calls pass false and take the
// recorded choice or else the first candidate, without timing.
// ---- depthwise 3x3 kernel configurations
// A choice is kept as a ConvKernel: fam 0 = register kernel (tile = strips
// per work item), fam 1 = band kernel (tile = rows | strips << 8, split =
// threads per workgroup).

// Band kernel geometry for bands of rb output rows and column tiles of ct
// strips (ct is capped at the strips of a row); false when the shape or
// the LDS size does not allow it.  threads == 0: one thread per strip and
// 4 channels of a tile, at most 512.
bool dw_band_config(DwArgs &a, int rb, int ct, int threads)
{
    a.band = 0;
    const int C = a.C, P = dw3_pixels();
    if (rb < 1 || rb > 64 || ct < 1 || ((int64_t)a.W * C) % 16 != 0 || (a.sh != 1 && a.sh != 2) ||
        (a.sw != 1 && a.sw != 2))
        return false;
    const int nstrip = (a.Wo + P - 1) / P;
    ct = std::min(ct, nstrip);
    const int nct = (nstrip + ct - 1) / ct;
    if (nct > 1 && C % 16 != 0)
        return false;   // column tiles start on 16-byte boundaries
    const int lcols = (ct * P - 1) * a.sw + 3;                  // LDS columns of a tile
    const int loff0 = nct > 1 ? 0 : (16 - (a.pl * C) % 16) % 16;  // image column 0 16-aligned
    const int64_t rowb = (int64_t)align_up((size_t)loff0 + (size_t)lcols * C, 16) + 16;
    const int64_t bytes = ((int64_t)(rb - 1) * a.sh + 3) * rowb;
    if (bytes > 65536)
        return false;
    const int64_t items = (int64_t)(C / 4) * ct;
    if (threads == 0)
        threads = (int)std::min<int64_t>(512, (items + 63) / 64 * 64);
    if (threads < 64 || threads > 512 || threads % 64 != 0)
        return false;
    const int nband = (a.Ho + rb - 1) / rb;
    if ((int64_t)a.N * nband * nct >= (int64_t(1) << 31) - 8)
        return false;
    a.band = 1;
    a.rb = rb;
    a.nband = nband;
    a.ct = ct;
    a.nct = nct;
    a.lcols = lcols;
    a.loff0 = loff0;
    a.lrs = (int32_t)rowb;
    a.lbytes = (int32_t)bytes;
    a.bthreads = threads;
    return true;
}

bool dw_apply(DwArgs &a, const ConvKernel &k)
{
    if (k.fam == 1)
        return dw_band_config(a, k.tile & 255, k.tile >> 8, k.split);
    const int P = dw3_pixels(), seg = k.tile;
    if (seg != 1 && seg != 2 && seg != 4)
        return false;
    const int64_t items = (int64_t)a.N * a.Ho * ((a.Wo + P * seg - 1) / (P * seg)) * (a.C / 8);
    if (items >= (int64_t(1) << 31))
        return false;
    a.band = 0;
    a.seg = seg;
    a.items = (int32_t)items;
    return true;
}

// Candidates: the register kernel (its default segment length first, the
// choice when nothing is timed), then band heights of 2, 4 and 8 rows with
// whole rows or 1/2, 1/4, 1/8 of a row per tile.
std::vector<ConvKernel> dw_candidates(const DwArgs &a, int seg_default)
{
    const int f_band = env_int("QNN_DWBAND", 1), f_seg = env_int("QNN_DW3T", 0);
    const int f_rb = env_int("QNN_DWRB", 0), f_ct = env_int("QNN_DWCT", 0), f_bt = env_int("QNN_DWBT", 0);
    DwArgs t = a;
    if (f_band != 0 && (f_rb > 0 || f_ct > 0 || f_bt > 0) &&
        dw_band_config(t, f_rb > 0 ? f_rb : 4, f_ct > 0 ? f_ct : (1 << 20), f_bt))
        return {{1, t.rb | (t.ct << 8), t.bthreads}};
    if (f_seg == 1 || f_seg == 2 || f_seg == 4)
        return {{0, f_seg, 1}};
    std::vector<ConvKernel> c = {{0, seg_default, 1}};
    if (f_band == 0)
        return c;
    for (int sg : {1, 2, 4})
        if (sg != seg_default && dw_apply(t, {0, sg, 1}))
            c.push_back({0, sg, 1});
    const int nstrip = (a.Wo + dw3_pixels() - 1) / dw3_pixels();
    for (int rb : {2, 4, 8})
        for (int div : {1, 2, 4, 8}) {
            const int ct = (nstrip + div - 1) / div;
            if (!dw_band_config(t, rb, ct, 0))
                continue;
            const ConvKernel k = {1, t.rb | (t.ct << 8), t.bthreads};
            bool dup = false;
            for (const ConvKernel &o : c)
                dup = dup || (o.fam == k.fam && o.tile == k.tile && o.split == k.split);
            if (!dup)
                c.push_back(k);
        }
    return c;
}

std::string dw_tune_key(const ConvDesc &d)
{
    bool zpw = false;
    for (int i = 0; i < d.wq.n; ++i)
        zpw = zpw || d.wq.zero_point[i] != 0;
    char buf[256];
    snprintf(buf, sizeof buf, "dw:x%d:n%d:h%d:w%d:c%d:r%d:s%d:st%dx%d:p%d,%d,%d,%d:y%d:q%d:z%d:l%d,%d", (int)d.xt,
             d.N, d.H, d.W, d.C, d.R, d.S, d.cp.stride_h, d.cp.stride_w, d.cp.pad_top, d.cp.pad_bottom,
             d.cp.pad_left, d.cp.pad_right, (int)d.yt, (int)d.rnd, (int)zpw, d.y_ldc, d.y_coff);
    return buf;
}

// Times the depthwise candidates on the plan's shape (constant-filled
// activations, cold caches as in autotune_conv) and returns the fastest.
qnn_status autotune_dw(const DwArgs &base, const std::vector<ConvKernel> &cands, hipStream_t st, ConvKernel *best)
{
    const size_t xb = align_up((size_t)base.N * base.H * base.W * base.C, 256);
    const size_t yb = align_up((size_t)base.N * base.Ho * base.Wo * base.y_ldc * (base.out_i32 ? 4 : 1), 256);
    void *buf = nullptr;
    hipError_t e = hipMalloc(&buf, xb + yb + 256);
    if (e != hipSuccess)
        return fail(QNN_ERR_ALLOC, "hipMalloc of %zu bytes for kernel tuning failed", xb + yb + 256);
    const size_t flush_bytes = size_t(320) << 20;
    void *flush = nullptr;
    if (hipMalloc(&flush, flush_bytes) != hipSuccess)
        flush = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    qnn_status s = QNN_OK;
    float best_ms = 1e30f;
    auto launch = [&](const DwArgs &t) { return t.band ? launch_depthwise3_band(t, st) : launch_depthwise3(t, st); };
    if ((e = hipMemsetAsync(buf, 0x35, xb + yb + 256, st)) != hipSuccess || (e = hipEventCreate(&e0)) != hipSuccess ||
        (e = hipEventCreate(&e1)) != hipSuccess) {
        s = hip_fail(e, "kernel tuning set-up");
    } else {
        for (const ConvKernel &k : cands) {
            DwArgs t = base;
            t.x = (const uint8_t *)buf;
            t.y = (char *)buf + xb;
            if (!dw_apply(t, k))
                continue;
            t.vec_store = t.band ? t.y_ldc % 4 == 0 && t.y_coff % 4 == 0 : t.y_ldc % 8 == 0 && t.y_coff % 8 == 0;
            if ((e = launch(t)) != hipSuccess)
                break;
            constexpr int kRuns = 5;
            float runs[kRuns];
            for (int r = 0; r < kRuns && e == hipSuccess; ++r) {
                if (flush && ((e = launch_cache_sweep(flush, flush_bytes, (int *)((char *)buf + xb + yb), st)) !=
                                  hipSuccess ||
                              (e = hipMemsetAsync(flush, r, size_t(16) << 20, st)) != hipSuccess))
                    break;
                if ((e = hipEventRecord(e0, st)) != hipSuccess || (e = launch(t)) != hipSuccess ||
                    (e = hipEventRecord(e1, st)) != hipSuccess || (e = hipEventSynchronize(e1)) != hipSuccess ||
                    (e = hipEventElapsedTime(&runs[r], e0, e1)) != hipSuccess)
                    break;
            }
            if (e != hipSuccess)
                break;
            std::sort(runs, runs + kRuns);
            if (runs[kRuns / 2] < best_ms) {
                best_ms = runs[kRuns / 2];
                *best = k;
            }
        }
        if (e != hipSuccess)
            s = hip_fail(e, "depthwise kernel tuning");
    }
    if (e0)
        (void)hipEventDestroy(e0);
    if (e1)
        (void)hipEventDestroy(e1);
    (void)hipStreamSynchronize(st);
    (void)hipFree(buf);
    if (flush)
        (void)hipFree(flush);
    return s;
}

qnn_status make_conv_plan(const ConvDesc &d, hipStream_t st, qnn_plan **out, bool tune = true)
{
    int32_t Ho, Wo, lo, hi;
    std::vector<int32_t> mult, shift;
    qnn_status s = validate_conv(d, &Ho, &Wo, &lo, &hi, &mult, &shift);
    if (s != QNN_OK)
        return s;
    std::vector<int32_t> bias_h;
    if ((s = read_bias(d.bias, d.K, st, &bias_h)) != QNN_OK)
        return s;
    const int64_t J = d.depthwise ? (int64_t)d.R * d.S : (int64_t)d.R * d.S * d.C;
    if ((s = check_overflow(d, J, bias_h)) != QNN_OK)
        return s;

    qnn_plan *p = new (std::nothrow) qnn_plan();
    if (!p)
        return fail(QNN_ERR_ALLOC, "out of host memory");
    const int32_t zpx = d.xq.zero_point[0];
    const int64_t M = (int64_t)d.N * Ho * Wo;

    if (d.depthwise) {
        p->kind = PLAN_DW;
        const int C = d.C, RS = d.R * d.S;
        // 3x3 layers run on the dot-product kernel; the general kernel's
        // weights are kept too (unaligned x, other filter sizes)
        // strips per work item: the longest segment that still leaves about
        // 16 waves per CU (QNN_DW3T=1|2|4 forces one)
        int seg = 1;
        {
            const int f = env_int("QNN_DW3T", 0);
            if (f == 1 || f == 2 || f == 4) {
                seg = f;
            } else {
                for (int t : {4, 2}) {
                    const int64_t it = (int64_t)d.N * Ho * ((Wo + dw3_pixels() * t - 1) / (dw3_pixels() * t)) * (C / 8);
                    if (it / 64 >= 16 * device_cus()) {
                        seg = t;
                        break;
                    }
                }
            }
        }
        const int64_t dw3_items =
            (int64_t)d.N * Ho * ((Wo + dw3_pixels() * seg - 1) / (dw3_pixels() * seg)) * (C / 8);
        const bool dw3 = d.R == 3 && d.S == 3 && d.cp.dil_h == 1 && d.cp.dil_w == 1 && C % 8 == 0 &&
                         (d.cp.stride_w == 1 || d.cp.stride_w == 2) && dw3_items < (int64_t(1) << 31) &&
                         (int64_t)d.N * d.H * d.W * C < (int64_t(1) << 31) &&
                         (int64_t)M * d.y_ldc * (d.yt == QNN_INT32 ? 4 : 1) < (int64_t(1) << 31) &&
                         env_int("QNN_DW3", 1) != 0;
        const int32_t zpx_l = d.xt == QNN_UINT8 ? zpx - 128 : zpx;
        const int32_t zpy = d.yt == QNN_INT32 ? 0 : d.yq.zero_point[0];
        const int32_t off8 = d.yt == QNN_INT8 ? 128 : 0;
        bool fast = d.yt != QNN_INT32 && d.rnd == QNN_ROUND_HALF_UP;
        for (int c = 0; c < C; ++c)
            if (shift[c] < 33 || shift[c] > 53)
                fast = false;
        bool zpw_any = false;
        for (int i = 0; i < d.wq.n; ++i)
            zpw_any = zpw_any || d.wq.zero_point[i] != 0;
        const size_t wq_bytes = align_up(sizeof(int32_t) * RS * C, 256);
        const size_t ch_bytes = align_up(sizeof(ChanRec) * C, 256);
        const size_t zw_bytes = align_up(sizeof(int32_t) * C, 256);
        const size_t wd_bytes = dw3 ? align_up(sizeof(uint32_t) * 3 * C, 256) : 0;
        const size_t ch3_bytes = dw3 ? ch_bytes : 0;
        const size_t total = wq_bytes + ch_bytes + zw_bytes + wd_bytes + ch3_bytes;
        hipError_t e = hipMalloc(&p->dev, total);
        if (e != hipSuccess) {
            free_plan(p);
            return fail(QNN_ERR_ALLOC, "hipMalloc of %zu bytes failed", total);
        }
        int32_t *wq = (int32_t *)p->dev;
        ChanRec *chan = (ChanRec *)((char *)p->dev + wq_bytes);
        int32_t *zpw_d = (int32_t *)((char *)p->dev + wq_bytes + ch_bytes);
        uint32_t *wd = dw3 ? (uint32_t *)((char *)zpw_d + zw_bytes) : nullptr;
        ChanRec *chan3 = dw3 ? (ChanRec *)((char *)zpw_d + zw_bytes + wd_bytes) : nullptr;
        std::vector<uint8_t> host(ch_bytes + zw_bytes, 0);
        std::vector<ChanRec> host3(dw3 ? C : 0);
        for (int c = 0; c < C; ++c) {
            const ChanRec r{mult[c], 0, 0, shift[c]};
            const int32_t z = d.wq.zero_point[d.wq.n == 1 ? 0 : c];
            std::memcpy(host.data() + sizeof(ChanRec) * c, &r, sizeof r);
            std::memcpy(host.data() + ch_bytes + sizeof(int32_t) * c, &z, sizeof z);
            if (dw3) {
                ChanRec r3{mult[c], 0, 0, shift[c]};
                if (fast) {
                    const int sh = shift[c] - 32;
                    r3.rndzp = (int32_t)((1LL << (sh - 1)) + (int64_t)(zpy + off8) * (1LL << sh));
                }
                host3[c] = r3;
            }
        }
        if ((e = hipMemcpyAsync(chan, host.data(), host.size(), hipMemcpyHostToDevice, st)) != hipSuccess ||
            (dw3 && (e = hipMemcpyAsync(chan3, host3.data(), sizeof(ChanRec) * C, hipMemcpyHostToDevice, st)) !=
                        hipSuccess) ||
            (e = launch_prep_dw(d.w, d.bias, RS, C, zpw_d, wq, chan, st)) != hipSuccess ||
            (dw3 && (e = launch_prep_dw3(d.w, d.bias, C, zpx_l, zpw_d, wd, chan3, st)) != hipSuccess) ||
            (e = hipStreamSynchronize(st)) != hipSuccess) {
            free_plan(p);
            return hip_fail(e, "depthwise plan preparation");
        }
        DwArgs &a = p->dw;
        a.wq = wq;
        a.chan = chan;
        a.N = d.N; a.H = d.H; a.W = d.W; a.C = d.C; a.Ho = Ho; a.Wo = Wo; a.R = d.R; a.S = d.S;
        a.sh = d.cp.stride_h; a.sw = d.cp.stride_w; a.pt = d.cp.pad_top; a.pl = d.cp.pad_left;
        a.dh = d.cp.dil_h; a.dw = d.cp.dil_w;
        a.zp_x = zpx;
        a.x_signed = d.xt == QNN_INT8;
        a.ydt = d.yt; a.lo = lo; a.hi = hi;
        a.zp_y = zpy;
        a.rounding = d.rnd;
        a.y_ldc = d.y_ldc; a.y_coff = d.y_coff;
        a.out_i32 = d.yt == QNN_INT32;
        a.wd = wd;
        a.zpw = zpw_d;
        a.flip4 = d.xt == QNN_UINT8 ? 0x80808080u : 0u;
        a.zp4 = 0x01010101u * (uint32_t)(uint8_t)zpx_l;
        a.zpw_any = zpw_any;
        a.fast_rq = fast;
        a.lo_off = lo + off8;
        a.hi_off = hi + off8;
        a.out_xor = off8 ? 0x80808080u : 0u;
        a.seg = seg;
        a.items = dw3 ? (int32_t)dw3_items : 0;
        // kernel choice among the register kernel's segment lengths and the
        // band kernel's band heights and column tiles, timed on this shape
        // (QNN_DWBAND=0 keeps the register kernel; QNN_DWRB=<rows>,
        // QNN_DWCT=<strips>, QNN_DWBT=<threads> force a band configuration)
        a.band = 0;
        if (dw3) {
            const std::vector<ConvKernel> cands = dw_candidates(a, seg);
            ConvKernel best = cands[0];
            if (cands.size() > 1 && M > 0 && tune && env_int("QNN_AUTOTUNE", 1) != 0) {
                const std::string key = dw_tune_key(d);
                if (!tune_lookup(key, cands, &best)) {
                    DwArgs t = a;
                    t.chan = chan3;
                    if ((s = autotune_dw(t, cands, st, &best)) != QNN_OK) {
                        free_plan(p);
                        return s;
                    }
                    tune_record(key, best);
                }
            }
            if (!dw_apply(a, best))
                a.band = 0;
        }
        p->dw3 = dw3;
        p->chan3 = chan3;
        char buf[128];
        if (dw3 && a.band)
            snprintf(buf, sizeof buf,
                     "depthwise band %dx%d stride %dx%d M=%lld C=%d rows=%d strips=%d threads=%d lds=%d", d.R, d.S,
                     a.sh, a.sw, (long long)M, C, a.rb, a.ct, a.bthreads, a.lbytes);
        else if (dw3)
            snprintf(buf, sizeof buf, "depthwise dot4 %dx%d stride %dx%d M=%lld C=%d seg=%d", d.R, d.S, a.sh, a.sw,
                     (long long)M, C, seg);
        else
            snprintf(buf, sizeof buf, "depthwise %dx%d stride %dx%d M=%lld C=%d", d.R, d.S, a.sh, a.sw,
                     (long long)M, C);
        p->desc = buf;
        *out = p;
        return QNN_OK;
    }

    p->kind = PLAN_CONV;
    // channel counts that are not a multiple of 4 are padded (with zp_x) to C4
    const int C4 = (d.C + 3) / 4 * 4;
    const int RS = d.R * d.S;
    const int64_t Jg = (int64_t)RS * C4;   // GEMM reduction length
    // weights are packed once for every kernel: rows padded to the largest
    // channel tile, the row stride to the largest K-step
    const int Kpad = (int)align_up(d.K, 256);
    const int Jpad = (int)align_up(Jg, 128);
    if ((int64_t)Kpad * Jpad >= (int64_t(1) << 31)) {
        free_plan(p);
        return fail(QNN_ERR_UNSUPPORTED, "packed weights of 2^31 bytes or more are not supported");
    }
    // the tap kernels gather one filter tap per K-step (C4 % BK == 0); the
    // LDS-direct one also needs the border classes for its padding fix-up
    BorderClasses bc;
    const bool term3 = [&] {
        for (int i = 0; i < d.wq.n; ++i)
            if (d.wq.zero_point[i] != 0)
                return true;
        return false;
    }();
    // tap-walk kernels: every K-step inside one filter tap (C4 % 64 == 0),
    // or a 1x1 filter over 16-byte pixels whose last K-step runs into the
    // next pixels (zero weights there)
    const bool one_tap = d.R == 1 && d.S == 1 && C4 % 16 == 0;
    const bool tap_ok = (C4 % 64 == 0 || one_tap) && d.R <= 16 && d.S <= 16;
    // row-pair mode of the LDS-direct kernel for small channel counts (the
    // 3-channel stems): two filter rows of S * C4 <= 32 bytes per K-step,
    // over a zero-point padded copy of the image
    const bool rowpack = !tap_ok && C4 * d.S <= 32 && d.R <= 32 && d.cp.dil_h == 1 && d.cp.dil_w == 1 && !term3 &&
                         env_int("QNN_ROWPACK", 1) != 0 && env_int("QNN_TILE", -1) < 0;
    const int npairs = (d.R + 1) / 2;
    const int Jr = npairs * 64;                      // row-pair reduction length
    const int Hp = std::max(d.H + d.cp.pad_top + d.cp.pad_bottom, (Ho - 1) * d.cp.stride_h + 2 * npairs);
    const int Wp = std::max(d.W + d.cp.pad_left + d.cp.pad_right, (Wo - 1) * d.cp.stride_w + (32 + C4 - 1) / C4);
    if (rowpack && (int64_t)d.N * Hp * Wp * C4 >= (int64_t(1) << 31)) {
        free_plan(p);
        return fail(QNN_ERR_UNSUPPORTED, "padded image of 2^31 bytes or more");
    }
    // the kernels index the channel-padded copy (C4 channels) in int32
    if (!rowpack && C4 != d.C && (int64_t)d.N * d.H * d.W * C4 >= (int64_t(1) << 31)) {
        free_plan(p);
        return fail(QNN_ERR_UNSUPPORTED, "channel-padded input of 2^31 bytes or more");
    }
    const bool dma_ok = tap_ok && border_classes(d, Ho, Wo, M, bc);
    const bool pcorr = dma_ok && bc.any && zpx != 0;
    const size_t ncls = pcorr ? bc.rmask.size() : 0;
    // legalisation (Sec. III-C): uint8 activations become int8 by x - 128
    const int32_t zpx_l = d.xt == QNN_UINT8 ? zpx - 128 : zpx;
    // 32-bit requantize in the epilogue when every channel allows it
    const int32_t zpy = d.yt == QNN_INT32 ? 0 : d.yq.zero_point[0];
    const int32_t off8 = d.yt == QNN_INT8 ? 128 : 0;
    bool fast = d.yt != QNN_INT32 && d.rnd == QNN_ROUND_HALF_UP;
    for (int k = 0; k < d.K; ++k)
        if (shift[k] < 33 || shift[k] > 53)
            fast = false;
    const bool staged = d.yt != QNN_INT32 && env_int("QNN_STAGED", 1) != 0;
    std::vector<ConvKernel> cands;
    if (rowpack) {
        const int f = env_int("QNN_DMA", -1);
        if (f >= 0 && f < DMA_COUNT && dma_split(f) == 1 && (!dma_short(f) || npairs <= dma_stages(f))) {
            cands.push_back({FAM_DMA, f});
        } else {
            for (int t : {DMA_128x128_S4, DMA_128x64_S4, DMA_64x128_S4, DMA_64x64_S4, DMA_128x64_S8, DMA_64x128_S8,
                          DMA_64x64_S8})
                cands.push_back({FAM_DMA, t});
            for (int t = DMA_64x128_R1; t < DMA_COUNT; ++t)
                if (dma_short(t) && npairs <= dma_stages(t))
                    cands.push_back({FAM_DMA, t});
        }
    } else {
        cands = conv_candidates(M, d.K, C4, (int)Jg, tap_ok, dma_ok, one_tap && C4 % 64 != 0);
    }

    const size_t wp_bytes = align_up((size_t)Kpad * Jpad, 256);
    const size_t wf_bytes = dma_ok ? wp_bytes : 0;
    const size_t wr_bytes = rowpack ? align_up((size_t)Kpad * Jr, 256) : 0;
    const size_t ch_bytes = align_up(sizeof(ChanRec) * Kpad, 256);
    const size_t zw_bytes = align_up(sizeof(int32_t) * Kpad, 256);
    const size_t pad_bytes = 256;
    const size_t pcls_bytes = pcorr ? align_up((size_t)M, 256) : 0;
    const size_t corr_bytes = pcorr ? align_up(sizeof(int32_t) * ncls * Kpad, 256) : 0;
    const size_t mask_bytes = pcorr ? align_up(sizeof(uint32_t) * 2 * ncls, 256) : 0;
    const size_t total =
        wp_bytes + wf_bytes + wr_bytes + ch_bytes + zw_bytes + pad_bytes + pcls_bytes + corr_bytes + mask_bytes;
    hipError_t e = hipMalloc(&p->dev, total);
    if (e != hipSuccess) {
        free_plan(p);
        return fail(QNN_ERR_ALLOC, "hipMalloc of %zu bytes failed", total);
    }
    int8_t *wp = (int8_t *)p->dev;
    int8_t *wf = dma_ok ? wp + wp_bytes : nullptr;
    int8_t *wr = rowpack ? wp + wp_bytes + wf_bytes : nullptr;
    ChanRec *chan = (ChanRec *)((char *)p->dev + wp_bytes + wf_bytes + wr_bytes);
    int32_t *zpw_d = (int32_t *)((char *)chan + ch_bytes);
    uint8_t *padbuf = (uint8_t *)zpw_d + zw_bytes;
    // channel records, weight zero points and the padding block (zp_x
    // bytes) in one upload
    std::vector<uint8_t> host(ch_bytes + zw_bytes + pad_bytes, 0);
    for (int k = 0; k < Kpad; ++k) {
        ChanRec r{0, 0, 0, 33};
        int32_t z = 0;
        if (k < d.K) {
            r.mult = mult[k];
            r.shift = shift[k];
            if (fast) {
                const int sh = shift[k] - 32;
                r.rndzp = (int32_t)((1LL << (sh - 1)) + (int64_t)(zpy + off8) * (1LL << sh));
            }
            z = d.wq.zero_point[d.wq.n == 1 ? 0 : k];
        }
        std::memcpy(host.data() + sizeof(ChanRec) * k, &r, sizeof r);
        std::memcpy(host.data() + ch_bytes + sizeof(int32_t) * k, &z, sizeof z);
    }
    std::memset(host.data() + ch_bytes + zw_bytes, (uint8_t)zpx, pad_bytes);
    uint8_t *pcls_d = padbuf + pad_bytes;
    int32_t *corr_d = (int32_t *)(pcls_d + pcls_bytes);
    uint32_t *mask_d = (uint32_t *)((char *)corr_d + corr_bytes);
    std::vector<uint32_t> masks;
    if (pcorr) {
        masks = bc.rmask;
        masks.insert(masks.end(), bc.cmask.begin(), bc.cmask.end());
    }
    if ((e = hipMemcpyAsync(chan, host.data(), host.size(), hipMemcpyHostToDevice, st)) != hipSuccess ||
        (e = launch_prep_conv(d.w, d.bias, d.K, RS, d.C, C4, Jpad, Kpad, zpx_l, wp, chan, zpw_d, st)) !=
            hipSuccess ||
        (wf && (e = launch_frag_pack(wp, Kpad, Jpad, wf, st)) != hipSuccess) ||
        (wr && (e = launch_rowpack_weights(d.w, d.K, d.R, d.S, d.C, C4, Kpad, Jr, wr, st)) != hipSuccess) ||
        (pcorr && ((e = hipMemcpyAsync(pcls_d, bc.pcls.data(), (size_t)M, hipMemcpyHostToDevice, st)) != hipSuccess ||
                   (e = hipMemcpyAsync(mask_d, masks.data(), sizeof(uint32_t) * masks.size(), hipMemcpyHostToDevice,
                                       st)) != hipSuccess ||
                   (e = launch_border_corr(wp, Kpad, Jpad, C4, d.S, RS, mask_d, mask_d + ncls, (int)ncls, zpx, corr_d,
                                           st)) != hipSuccess)) ||
        (e = hipStreamSynchronize(st)) != hipSuccess) {
        free_plan(p);
        return hip_fail(e, "conv plan preparation");
    }

    ConvArgs &a = p->conv;
    a.wp = wp;
    a.wf = wf;
    a.chan = chan;
    a.zpw = zpw_d;
    a.padbuf = padbuf;
    a.N = d.N; a.H = d.H; a.W = d.W; a.C = C4; a.Ho = Ho; a.Wo = Wo; a.R = d.R; a.S = d.S;
    a.sh = d.cp.stride_h; a.sw = d.cp.stride_w; a.pt = d.cp.pad_top; a.pl = d.cp.pad_left;
    a.dh = d.cp.dil_h; a.dw = d.cp.dil_w;
    a.K = d.K; a.Kpad = Kpad; a.J = (int)Jg; a.Jpad = Jpad; a.M = (int)M;
    p->C_in = d.C;
    p->pad_zp = (uint8_t)zpx;
    p->y_scale = d.yt == QNN_INT32 ? 1.0f : d.yq.scale[0];
    p->y_zp = d.yt == QNN_INT32 ? 0 : d.yq.zero_point[0];
    p->y_dt = d.yt;
    a.flip4 = d.xt == QNN_UINT8 ? 0x80808080u : 0u;
    a.ydt = d.yt;
    a.lo = lo; a.hi = hi;
    a.zp_y = d.yt == QNN_INT32 ? 0 : d.yq.zero_point[0];
    a.rounding = d.rnd;
    a.y_ldc = d.y_ldc; a.y_coff = d.y_coff;
    a.vec_store = (d.y_ldc % 4 == 0) && (d.y_coff % 4 == 0);
    p->avec = gather_width(C4);
    p->mode = d.yt == QNN_INT32 ? OUT_INT32 : OUT_REQUANT;
    a.mode = p->mode;
    a.fast_rq = fast;
    a.lo_off = lo + off8;
    a.hi_off = hi + off8;
    a.out_xor = off8 ? 0x80808080u : 0u;
    a.staged = staged;
    a.zp4 = 0x01010101u * (uint32_t)(uint8_t)zpx_l;
    const int32_t *pcorr_tab = pcorr ? corr_d : nullptr;
    const uint8_t *pcls_tab = pcorr ? pcls_d : nullptr;
    a.chan_in_lds = (size_t)Kpad * sizeof(ChanRec) <= 64 * 1024;
    make_divider((uint32_t)Wo, a.mWo, a.sWo);
    make_divider((uint32_t)Ho, a.mHo, a.sHo);
    p->term3 = term3;
    p->ws_asum_bytes = term3 ? align_up((size_t)M * sizeof(int32_t), 256) : 0;
    p->ws_xpad_bytes = rowpack ? align_up((size_t)d.N * Hp * Wp * C4, 256)
                               : C4 != d.C ? align_up((size_t)d.N * d.H * d.W * C4, 256) : 0;
    p->rowpack = rowpack;
    p->H_in = d.H; p->W_in = d.W; p->pt_in = d.cp.pad_top; p->pl_in = d.cp.pad_left;
    if (rowpack) {
        // the kernel sees the padded image, unpadded, with row pairs as taps
        a.wp = wr;
        a.Jpad = Jr;
        a.J = Jr;
        a.H = Hp; a.W = Wp;
        a.pt = 0; a.pl = 0;
        a.R = npairs; a.S = 1;
        a.rowpack = 1;
        a.row_bytes = Wp * C4;
    }
    p->ws_bytes = p->ws_asum_bytes + p->ws_xpad_bytes;

    // the window kernel joins the candidates of the shapes it serves when
    // its LDS fits; QNN_HALO=4|8 forces it (if eligible), -2 leaves it out
    if (!rowpack && dma_ok) {
        const int f_halo = env_int("QNN_HALO", -1);
        const int f_wave = env_int("QNN_WAVE", -1);
        const bool other_forced = env_int("QNN_DMA", -1) >= 0 || env_int("QNN_TAP", -1) >= 0 ||
                                  env_int("QNN_TILE", -1) >= 0 ||
                                  f_wave == 1 || f_wave == 2 || f_wave == 4 || f_wave == 8;
        std::vector<ConvKernel> hk;
        for (int nw : {8, 4}) {
            const size_t lds = halo_lds_bytes(a, nw);
            if (lds && lds <= (size_t)device_lds_per_block() && (f_halo < 0 || f_halo == nw))
                hk.push_back({FAM_HALO, nw});
        }
        if (f_halo == 4 || f_halo == 8) {
            if (!hk.empty())
                cands = hk;
        } else if (f_halo != -2 && !other_forced) {
            cands.insert(cands.end(), hk.begin(), hk.end());
        }
        // the streaming window kernel likewise: QNN_WIN=<cfg> forces one
        // configuration (if eligible), -2 leaves the family out
        const int f_win = env_int("QNN_WIN", -1);
        std::vector<ConvKernel> wk;
        for (int c = 0; c < win_count(); ++c) {
            const size_t lds = win_lds_bytes(a, c);
            if (lds && lds <= (size_t)device_lds_per_block() && (f_win < 0 || f_win == c))
                wk.push_back({FAM_WIN, c});
        }
        if (f_win >= 0) {
            if (!wk.empty())
                cands = wk;
        } else if (f_win != -2 && f_halo < 0 && !other_forced) {
            cands.insert(cands.end(), wk.begin(), wk.end());
        }
    }

    // kernel choice: the candidates are timed on this very shape (the
    // weights and tables are real, the activations a constant fill) and
    // the fastest is kept; every candidate computes the same bytes
    ConvKernel best = cands[0];
    if (cands.size() > 1 && M > 0 && env_int("QNN_AUTOTUNE", 1) != 0) {
        const std::string key = tune_key(d, term3, ncls, fast);
        if (!tune_lookup(key, cands, &best) && tune) {
            if ((s = autotune_conv(a, cands, p->avec, term3, pcorr_tab, pcls_tab, st, &best)) != QNN_OK) {
                free_plan(p);
                return s;
            }
            tune_record(key, best);
        }
    }
    p->ker = best;
    set_tiling(a, best, p->avec, pcorr_tab, pcls_tab);
    if ((int64_t)a.ntiles < 0) {
        free_plan(p);
        return fail(QNN_ERR_UNSUPPORTED, "too many output tiles");
    }
    if (a.ksplit > 1) {
        const TileShape st_ = kernel_shape(best);
        p->ws_cnt_bytes = align_up((size_t)a.ntiles * sizeof(int32_t), 256);
        p->ws_part_bytes = (size_t)a.ntiles * a.ksplit * st_.tc * st_.tp * sizeof(int32_t);
        p->ws_bytes += p->ws_cnt_bytes + p->ws_part_bytes;
    }
    const TileShape ts = kernel_shape(best);
    static const char *fam_name[] = {"conv_mfma", "conv_tap", "conv_dma", "conv_wave", "conv_halo", "conv_window"};
    char buf[200];
    if (best.fam == FAM_GATHER)
        snprintf(buf, sizeof buf,
                 "conv_mfma tile=%dx%dx%d gather=%d tiles=%d grid=%d term3=%d cpad=%d M=%lld K=%d J=%lld cands=%d",
                 ts.tc, ts.tp, ts.bk, p->avec, a.ntiles, a.nblocks, (int)term3, C4 != d.C, (long long)M, d.K,
                 (long long)Jg, (int)cands.size());
    else
        snprintf(buf, sizeof buf,
                 "%s tile=%dx%dx%d threads=%d stages=%d%s tiles=%d term3=%d border=%d M=%lld K=%d J=%lld cands=%d",
                 fam_name[best.fam], ts.tc, ts.tp, ts.bk,
                 best.fam == FAM_DMA    ? dma_threads(best.tile)
                 : best.fam == FAM_WAVE ? wave_threads(best.tile)
                 : best.fam == FAM_HALO ? best.tile * 64
                 : best.fam == FAM_WIN  ? win_threads(best.tile)
                                        : tap_threads(best.tile),
                 best.fam == FAM_DMA ? dma_stages(best.tile) : best.fam == FAM_WAVE ? 4 : best.fam == FAM_HALO ? 1 : 2,
                 best.fam == FAM_DMA && dma_short(best.tile) ? "s" : "", a.ntiles, (int)term3,
                 (int)ncls, (long long)M, d.K, (long long)Jg, (int)cands.size());
    if (best.fam == FAM_WAVE) {
        const size_t n = strlen(buf);
        snprintf(buf + n, sizeof buf - n, " split=%d", best.tile);
    } else if (best.fam == FAM_DMA && best.split > 1) {
        const size_t n = strlen(buf);
        snprintf(buf + n, sizeof buf - n, " ksplit=%d", best.split);
    } else if (best.fam == FAM_WIN) {
        const size_t n = strlen(buf);
        snprintf(buf + n, sizeof buf - n, " cfg=%d", best.tile);
    } else if (best.fam == FAM_HALO) {
        const int lay = halo_layout(a, best.tile);
        const size_t n = strlen(buf);
        snprintf(buf + n, sizeof buf - n, " sep=%d", lay);
    }
    p->desc = buf;
    *out = p;
    return QNN_OK;
}

// Runs a plan with its workspace in two parts: `cnt` holds the split
// reduction's arrival counters (zero between runs), `ws` the window sums,
// the padded input copy and the partial sums, in that order.  A workspace
// of qnn_plan_workspace_size bytes holds the counters first, then the rest.
qnn_status run_plan_at(const qnn_plan *p, hipStream_t st, const void *x, void *y, void *cnt, void *ws,
                       const void *res = nullptr)
{
    if (p->fused != (res != nullptr))
        return fail(p->fused ? QNN_ERR_NULL : QNN_ERR_UNSUPPORTED,
                    p->fused ? "plan_run: the plan adds a residual; run it with qnn_plan_run_residual and a residual"
                             : "plan_run: a residual was given to a plan without a fused add");
    switch (p->kind) {
    case PLAN_CONV: {
        ConvArgs a = p->conv;
        if (a.M == 0)
            return QNN_OK;
        if (!x || !y)
            return fail(QNN_ERR_NULL, "plan_run: x or y is NULL");
        a.x = (const uint8_t *)x;
        a.y = y;
        if (res) {
            a.res = (const uint8_t *)res;
            a.res_vec = ((uintptr_t)res & 15) == 0 && a.r_ldc % 16 == 0 && a.r_coff % 16 == 0;
        }
        if (p->ws_bytes) {
            if (!ws || (p->ws_cnt_bytes && !cnt))
                return fail(QNN_ERR_NULL, "plan_run: the plan needs a workspace");
            a.asum = p->term3 ? (const int32_t *)ws : nullptr;
            if (p->ws_cnt_bytes) {
                a.cnt = (int32_t *)cnt;
                a.part = (int32_t *)((char *)ws + p->ws_asum_bytes + p->ws_xpad_bytes);
            }
        }
        hipError_t e;
        if (p->ws_xpad_bytes) {
            uint8_t *xp = (uint8_t *)ws + p->ws_asum_bytes;
            if (p->rowpack) {
                if ((e = launch_pad_image(a.x, a.N, p->H_in, p->W_in, p->C_in, a.H, a.W, a.C, p->pt_in, p->pl_in,
                                          p->pad_zp, xp, st)) != hipSuccess)
                    return hip_fail(e, "image padding launch");
            } else {
                const long long pixels = (long long)a.N * a.H * a.W;
                if ((e = launch_pad_channels(a.x, xp, pixels, p->C_in, a.C, p->pad_zp, st)) != hipSuccess)
                    return hip_fail(e, "channel padding launch");
            }
            a.x = xp;
            x = xp;
        }
        if (((uintptr_t)x & 15) != 0 && p->avec == 16)
            return fail(QNN_ERR_UNSUPPORTED, "plan_run: x must be 16-byte aligned for C %% 16 == 0");
        if (((uintptr_t)x & 3) != 0 && p->avec == 4)
            return fail(QNN_ERR_UNSUPPORTED, "plan_run: x must be 4-byte aligned for C %% 4 == 0");
        if (((uintptr_t)x & 7) != 0 && p->avec == 8)
            return fail(QNN_ERR_UNSUPPORTED, "plan_run: x must be 8-byte aligned for C %% 8 == 0");
        if (a.vec_store && ((uintptr_t)y & (p->mode == OUT_INT32 ? 15 : 3)) != 0)
            a.vec_store = 0;
        // whole-row 16-byte stores need a 16-byte aligned row start for every pixel
        if (a.staged && (((uintptr_t)y & 15) != 0 || a.y_ldc % 16 != 0 || a.y_coff % 16 != 0))
            a.staged = 0;
        if (a.res && !a.staged)
            return fail(QNN_ERR_UNSUPPORTED, "plan_run_residual: y must be 16-byte aligned for the fused add");
        if (p->term3 && (e = launch_window_sums(a, (int32_t *)a.asum, st)) != hipSuccess)
            return hip_fail(e, "window-sum launch");
        if ((e = launch_conv_kernel(a, p->ker, p->avec, st)) != hipSuccess)
            return hip_fail(e, "conv launch");
        return QNN_OK;
    }
    case PLAN_DW: {
        DwArgs a = p->dw;
        if ((int64_t)a.N * a.Ho * a.Wo == 0)
            return QNN_OK;
        if (!x || !y)
            return fail(QNN_ERR_NULL, "plan_run: x or y is NULL");
        a.x = (const uint8_t *)x;
        a.y = y;
        hipError_t e;
        if (p->dw3 && a.band && ((uintptr_t)x & 15) == 0) {
            a.chan = p->chan3;
            a.vec_store = ((uintptr_t)y & 3) == 0 && a.y_ldc % 4 == 0 && a.y_coff % 4 == 0;
            e = launch_depthwise3_band(a, st);
        } else if (p->dw3 && ((uintptr_t)x & 7) == 0) {
            a.chan = p->chan3;
            a.vec_store = ((uintptr_t)y & 7) == 0 && a.y_ldc % 8 == 0 && a.y_coff % 8 == 0;
            e = launch_depthwise3(a, st);
        } else {
            e = launch_depthwise(a, st);
        }
        return e == hipSuccess ? QNN_OK : hip_fail(e, "depthwise launch");
    }
    case PLAN_REQ: {
        ReqArgs a = p->req;
        if (a.count == 0)
            return QNN_OK;
        if (!x || !y)
            return fail(QNN_ERR_NULL, "plan_run: x or y is NULL");
        a.x = x;
        a.y = y;
        const bool aligned = ((uintptr_t)x & 15) == 0 && ((uintptr_t)y & 15) == 0;
        hipError_t e = launch_requantize(a, p->xdt, p->ydt, aligned, st);
        return e == hipSuccess ? QNN_OK : hip_fail(e, "requantize launch");
    }
    }
    return fail(QNN_ERR_UNSUPPORTED, "unknown plan kind");
}

qnn_status run_plan(const qnn_plan *p, hipStream_t st, const void *x, void *y, void *ws, const void *res = nullptr)
{
    if (!ws)
        ws = p->ws_own;
    char *base = (char *)ws;
    return run_plan_at(p, st, x, y, base, base ? base + p->ws_cnt_bytes : nullptr, res);
}

qnn_status alloc_ws(qnn_plan *p)
{
    if (!p->ws_bytes)
        return QNN_OK;
    if (hipMalloc(&p->ws_own, p->ws_bytes) != hipSuccess)
        return fail(QNN_ERR_ALLOC, "hipMalloc of a %zu-byte workspace failed", p->ws_bytes);
    // split reductions need their arrival counters at zero before the first run
    if (p->ws_cnt_bytes && hipMemset(p->ws_own, 0, p->ws_bytes) != hipSuccess)
        return fail(QNN_ERR_HIP, "zeroing the workspace failed");
    return QNN_OK;
}

qnn_status one_shot(const ConvDesc &d, hipStream_t st, const void *x, void *y)
{
    {
        // empty input: validate the arguments, then nothing to do
        int32_t Ho, Wo, lo, hi;
        std::vector<int32_t> mult, shift;
        qnn_status s = validate_conv(d, &Ho, &Wo, &lo, &hi, &mult, &shift);
        if (s != QNN_OK || d.N == 0)
            return s;
    }
    qnn_plan *p = nullptr;
    qnn_status s = make_conv_plan(d, st, &p, false);
    if (s != QNN_OK)
        return s;
    if ((s = alloc_ws(p)) == QNN_OK && (s = run_plan(p, st, x, y, nullptr)) == QNN_OK) {
        const hipError_t e = hipStreamSynchronize(st);
        if (e != hipSuccess)
            s = hip_fail(e, "stream synchronize");
    }
    free_plan(p);
    return s;
}

ConvDesc conv_desc(qnn_dtype xt, int32_t N, int32_t H, int32_t W, int32_t C, qnn_qparams xq, const int8_t *w,
                   int32_t K, int32_t R, int32_t S, qnn_qparams wq, const int32_t *bias, qnn_conv_params cp,
                   qnn_dtype yt, qnn_qparams yq, qnn_clamp act, qnn_rounding rnd, int32_t y_ldc, int32_t y_coff,
                   bool dw)
{
    return ConvDesc{xt, N, H, W, C, xq, w, K, R, S, wq, bias, cp, yt, yq, act, rnd, y_ldc, y_coff, dw};
}

ConvDesc dense_desc(qnn_dtype xt, int32_t M, int32_t Kd, qnn_qparams xq, const int8_t *w, int32_t Nd,
                    qnn_qparams wq, const int32_t *bias, qnn_dtype yt, qnn_qparams yq, qnn_clamp act,
                    qnn_rounding rnd, int32_t y_ldc)
{
    // dense is the 1x1 conv of a [1][1][M][Kd] "image"
    const qnn_conv_params cp{1, 1, 0, 0, 0, 0, 1, 1};
    return ConvDesc{xt, M > 0 ? 1 : 0, 1, M > 0 ? M : 1, Kd, xq, w, Nd, 1, 1, wq, bias, cp, yt, yq, act, rnd,
                    y_ldc, 0, false};
}

qnn_status make_req_plan(qnn_dtype xt, int64_t count, int32_t channels, qnn_qparams xq, qnn_dtype yt,
                         qnn_qparams yq, qnn_clamp act, qnn_rounding rnd, hipStream_t st, bool upload,
                         qnn_plan **out)
{
    if (xt != QNN_UINT8 && xt != QNN_INT8 && xt != QNN_INT32)
        return fail(QNN_ERR_DTYPE, "requantize: unknown input dtype");
    if (yt != QNN_UINT8 && yt != QNN_INT8 && yt != QNN_INT32)
        return fail(QNN_ERR_DTYPE, "requantize: unknown output dtype");
    if (rnd < QNN_ROUND_HALF_UP || rnd > QNN_ROUND_TWO_STAGE)
        return fail(QNN_ERR_QPARAM, "requantize: unknown rounding %d", (int)rnd);
    if (count < 0 || channels < 1 || count % channels != 0)
        return fail(QNN_ERR_SHAPE, "requantize: count must be a non-negative multiple of channels >= 1");
    qnn_status s;
    if ((s = check_qparams(xq, "x qparams", channels, xt, false)) != QNN_OK)
        return s;
    if ((s = check_qparams(yq, "y qparams", channels, yt, false)) != QNN_OK)
        return s;
    if (xt == QNN_INT32)
        for (int i = 0; i < xq.n; ++i)
            if (xq.zero_point[i] != 0)
                return fail(QNN_ERR_QPARAM, "requantize: int32 input requires zero point 0");
    int32_t lo, hi;
    if ((s = out_bounds(yt, act, &lo, &hi)) != QNN_OK)
        return s;
    const bool perch = xq.n > 1 || yq.n > 1;
    const int nc = perch ? channels : 1;
    std::vector<int32_t> tab(4 * (size_t)nc);
    for (int c = 0; c < nc; ++c) {
        const int ci = xq.n == 1 ? 0 : c, co = yq.n == 1 ? 0 : c;
        const double M = (double)xq.scale[ci] / (double)yq.scale[co];
        int32_t m, n;
        if (!derive_multiplier(M, &m, &n))
            return fail(QNN_ERR_QPARAM, "requantize: multiplier %g is out of range", M);
        tab[4 * c] = m;
        tab[4 * c + 1] = n > 63 ? 63 : n;
        tab[4 * c + 2] = xq.zero_point[ci];
        tab[4 * c + 3] = yq.zero_point[co];
    }
    qnn_plan *p = new (std::nothrow) qnn_plan();
    if (!p)
        return fail(QNN_ERR_ALLOC, "out of host memory");
    p->kind = PLAN_REQ;
    p->xdt = xt;
    p->ydt = yt;
    ReqArgs &a = p->req;
    a.count = count;
    a.channels = channels;
    a.mult = tab[0]; a.shift = tab[1]; a.zp_in = tab[2]; a.zp_out = tab[3];
    a.lo = lo; a.hi = hi; a.rounding = rnd;
    a.tab = nullptr;
    if (perch) {
        if (!upload) {
            free_plan(p);
            return fail(QNN_ERR_UNSUPPORTED, "internal: per-channel requantize needs an upload");
        }
        hipError_t e = hipMalloc(&p->dev, tab.size() * sizeof(int32_t));
        if (e != hipSuccess) {
            free_plan(p);
            return fail(QNN_ERR_ALLOC, "hipMalloc failed");
        }
        if ((e = hipMemcpyAsync(p->dev, tab.data(), tab.size() * sizeof(int32_t), hipMemcpyHostToDevice, st)) !=
                hipSuccess ||
            (e = hipStreamSynchronize(st)) != hipSuccess) {
            free_plan(p);
            return hip_fail(e, "requantize table upload");
        }
        a.tab = (const int32_t *)p->dev;
    }
    char buf[96];
    snprintf(buf, sizeof buf, "requantize %s->%s count=%lld channels=%d perch=%d", dtype_name(xt), dtype_name(yt),
             (long long)count, channels, (int)perch);
    p->desc = buf;
    *out = p;
    return QNN_OK;
}

// ---------------------------------------------------------------- uint8 weights
//
// Weights given as asymmetric uint8 are legalised once, when the plan is
// created, the way Sec. III-C legalises activations: w' = w - 128 (each
// byte XOR 0x80, read as int8) and zp_w' = zp_w - 128, which leaves every
// (w - zp_w), hence the accumulator, unchanged.  The int8 copy lives in a
// temporary device buffer for the plan's preparation kernels only.
struct LegalWeights {
    void *dev = nullptr;
    std::vector<int32_t> zp;
    qnn_qparams q{};
    ~LegalWeights()
    {
        if (dev)
            (void)hipFree(dev);
    }
};

qnn_status legalize_weights(const void *w, qnn_dtype wt, size_t n, const qnn_qparams &wq, int32_t channels,
                            hipStream_t st, LegalWeights *out, const int8_t **w8, qnn_qparams *wq8)
{
    if (wt == QNN_INT8) {
        *w8 = (const int8_t *)w;
        *wq8 = wq;
        return QNN_OK;
    }
    if (wt != QNN_UINT8)
        return fail(QNN_ERR_DTYPE, "weights must be int8 or uint8");
    qnn_status s = check_qparams(wq, "w qparams", channels, QNN_UINT8, true);
    if (s != QNN_OK)
        return s;
    if (!w)
        return fail(QNN_ERR_NULL, "weight pointer is NULL");
    out->zp.assign(wq.zero_point, wq.zero_point + wq.n);
    for (int32_t &z : out->zp)
        z -= 128;
    out->q = qnn_qparams{wq.scale, out->zp.data(), wq.n};
    hipError_t e;
    if (n && (e = hipMalloc(&out->dev, n)) != hipSuccess)
        return fail(QNN_ERR_ALLOC, "hipMalloc of %zu bytes for the legalised weights failed", n);
    if (n && (e = launch_flip_bytes((const uint8_t *)w, (uint8_t *)out->dev, n, st)) != hipSuccess)
        return hip_fail(e, "weight legalisation launch");
    *w8 = (const int8_t *)out->dev;
    *wq8 = out->q;
    return QNN_OK;
}

// ---------------------------------------------------------------- allocation-free runs
//
// qnn_plan_run_noalloc takes its workspace from this file-scope device
// array instead of memory the caller or the plan allocated: the first
// kScratchCntBytes hold the split reduction's arrival counters (zero
// between runs: every split kernel resets the counters it used), the rest
// the window sums, the padded input copy and the partial sums of one run.
// In host code `scratch` names a host-side stand-in; its device address is
// taken once per device (hipGetSymbolAddress) and only that address is
// passed to kernels.
constexpr size_t kScratchBytes = size_t(64) << 20;
constexpr size_t kScratchCntBytes = size_t(1) << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

__global__ void __launch_bounds__(256) zero_words_kernel(uint32_t *p, size_t n)
{
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

std::mutex g_scratch_mu;
char *g_scratch[kMaxDevices] = {};

// The device address of `scratch` on the current device.  On the first
// call for a device its counter region is cleared by a kernel on `st` (not
// a memset, so that the clear is stream-ordered like the runs after it).
qnn_status scratch_for_device(hipStream_t st, char **out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices)
        return fail(QNN_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
    std::lock_guard<std::mutex> g(g_scratch_mu);
    if (!g_scratch[dev]) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        if ((e = hipStreamIsCapturing(st, &cs)) != hipSuccess)
            return hip_fail(e, "hipStreamIsCapturing");
        if (cs != hipStreamCaptureStatusNone)
            return fail(QNN_ERR_UNSUPPORTED,
                        "plan_run_noalloc: the first call on a device sets up its scratch and must not be captured");
        void *ptr = nullptr;
        if ((e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch))) != hipSuccess || !ptr)
            return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "hipGetSymbolAddress of the scratch array");
        hipLaunchKernelGGL(zero_words_kernel, dim3(256), dim3(256), 0, st, (uint32_t *)ptr,
                           kScratchCntBytes / sizeof(uint32_t));
        if ((e = hipGetLastError()) != hipSuccess)
            return hip_fail(e, "scratch clear launch");
        g_scratch[dev] = (char *)ptr;
    }
    *out = g_scratch[dev];
    return QNN_OK;
}

}  // namespace

// ==================================================================== ABI

extern "C" {

int32_t qnn_abi_version(void) { return QNN_ABI_VERSION; }

const char *qnn_last_error(void) { return g_last_error.c_str(); }

const char *qnn_status_string(qnn_status s)
{
    switch (s) {
    case QNN_OK: return "QNN_OK";
    case QNN_ERR_NULL: return "QNN_ERR_NULL";
    case QNN_ERR_SHAPE: return "QNN_ERR_SHAPE";
    case QNN_ERR_DTYPE: return "QNN_ERR_DTYPE";
    case QNN_ERR_QPARAM: return "QNN_ERR_QPARAM";
    case QNN_ERR_OVERFLOW: return "QNN_ERR_OVERFLOW";
    case QNN_ERR_UNSUPPORTED: return "QNN_ERR_UNSUPPORTED";
    case QNN_ERR_HIP: return "QNN_ERR_HIP";
    case QNN_ERR_ALLOC: return "QNN_ERR_ALLOC";
    }
    return "QNN_ERR_?";
}

qnn_status qnn_quantize_multiplier(double M, int32_t *mult, int32_t *shift)
{
    if (!mult || !shift)
        return fail(QNN_ERR_NULL, "quantize_multiplier: NULL output pointer");
    if (!derive_multiplier(M, mult, shift))
        return fail(QNN_ERR_QPARAM, "multiplier %g is negative, not finite or too large", M);
    return QNN_OK;
}

qnn_status qnn_conv2d(void *stream, const void *x, qnn_dtype x_dtype, int32_t N, int32_t H, int32_t W, int32_t C,
                      qnn_qparams x_q, const int8_t *w, int32_t K, int32_t R, int32_t S, qnn_qparams w_q,
                      const int32_t *bias, qnn_conv_params conv, void *y, qnn_dtype y_dtype, qnn_qparams y_q,
                      qnn_clamp act, qnn_rounding rounding, int32_t y_ldc, int32_t y_coff)
{
    const ConvDesc d = conv_desc(x_dtype, N, H, W, C, x_q, w, K, R, S, w_q, bias, conv, y_dtype, y_q, act,
                                 rounding, y_ldc, y_coff, false);
    if (N > 0 && (!x || !y))
        return fail(QNN_ERR_NULL, "conv2d: x or y is NULL");
    return one_shot(d, (hipStream_t)stream, x, y);
}

qnn_status qnn_depthwise_conv2d(void *stream, const void *x, qnn_dtype x_dtype, int32_t N, int32_t H, int32_t W,
                                int32_t C, qnn_qparams x_q, const int8_t *w, int32_t R, int32_t S, qnn_qparams w_q,
                                const int32_t *bias, qnn_conv_params conv, void *y, qnn_dtype y_dtype,
                                qnn_qparams y_q, qnn_clamp act, qnn_rounding rounding, int32_t y_ldc,
                                int32_t y_coff)
{
    const ConvDesc d = conv_desc(x_dtype, N, H, W, C, x_q, w, C, R, S, w_q, bias, conv, y_dtype, y_q, act,
                                 rounding, y_ldc, y_coff, true);
    if (N > 0 && (!x || !y))
        return fail(QNN_ERR_NULL, "depthwise_conv2d: x or y is NULL");
    return one_shot(d, (hipStream_t)stream, x, y);
}

qnn_status qnn_dense(void *stream, const void *x, qnn_dtype x_dtype, int32_t M, int32_t Kd, qnn_qparams x_q,
                     const int8_t *w, int32_t Nd, qnn_qparams w_q, const int32_t *bias, void *y, qnn_dtype y_dtype,
                     qnn_qparams y_q, qnn_clamp act, qnn_rounding rounding, int32_t y_ldc)
{
    if (M < 0)
        return fail(QNN_ERR_SHAPE, "dense: M must be >= 0");
    const ConvDesc d = dense_desc(x_dtype, M, Kd, x_q, w, Nd, w_q, bias, y_dtype, y_q, act, rounding, y_ldc);
    if (M > 0 && (!x || !y))
        return fail(QNN_ERR_NULL, "dense: x or y is NULL");
    return one_shot(d, (hipStream_t)stream, x, y);
}

qnn_status qnn_requantize(void *stream, const void *x, qnn_dtype x_dtype, int64_t count, int32_t channels,
                          qnn_qparams x_q, void *y, qnn_dtype y_dtype, qnn_qparams y_q, qnn_clamp act,
                          qnn_rounding rounding)
{
    hipStream_t st = (hipStream_t)stream;
    qnn_plan *p = nullptr;
    qnn_status s = make_req_plan(x_dtype, count, channels, x_q, y_dtype, y_q, act, rounding, st, true, &p);
    if (s != QNN_OK)
        return s;
    if (count > 0 && (!x || !y)) {
        free_plan(p);
        return fail(QNN_ERR_NULL, "requantize: x or y is NULL");
    }
    s = run_plan(p, st, x, y, nullptr);
    if (s == QNN_OK && p->dev) {
        const hipError_t e = hipStreamSynchronize(st);
        if (e != hipSuccess)
            s = hip_fail(e, "stream synchronize");
    }
    free_plan(p);
    return s;
}

qnn_status qnn_pool2d(void *stream, const void *x, qnn_dtype dtype, int32_t N, int32_t H, int32_t W, int32_t C,
                      int32_t R, int32_t S, qnn_conv_params pool, qnn_pool_mode mode, int32_t count_pad,
                      int32_t zero_point, void *y, qnn_rounding rounding)
{
    if (dtype != QNN_UINT8 && dtype != QNN_INT8)
        return fail(QNN_ERR_DTYPE, "pool2d: dtype must be uint8 or int8");
    if (mode != QNN_POOL_AVG && mode != QNN_POOL_MAX)
        return fail(QNN_ERR_UNSUPPORTED, "pool2d: unknown mode %d", (int)mode);
    const bool avg = mode == QNN_POOL_AVG;
    if (avg && rounding != QNN_ROUND_HALF_UP && rounding != QNN_ROUND_HALF_AWAY)
        return fail(QNN_ERR_QPARAM, "pool2d: average pooling rounds HALF_UP or HALF_AWAY (got %d)", (int)rounding);
    if (avg && count_pad != 0 && count_pad != 1)
        return fail(QNN_ERR_SHAPE, "pool2d: count_pad must be 0 or 1");
    const bool sgn = dtype == QNN_INT8;
    if (avg && count_pad && (zero_point < (sgn ? -128 : 0) || zero_point > (sgn ? 127 : 255)))
        return fail(QNN_ERR_QPARAM, "pool2d: zero point %d outside the %s range", zero_point, dtype_name(dtype));
    if (N < 0 || H < 1 || W < 1 || C < 1 || R < 1 || S < 1)
        return fail(QNN_ERR_SHAPE, "pool2d: sizes must be positive (N >= 0)");
    if (pool.stride_h < 1 || pool.stride_w < 1 || pool.dil_h != 1 || pool.dil_w != 1)
        return fail(QNN_ERR_SHAPE, "pool2d: strides must be >= 1 and dilations 1");
    if (pool.pad_top < 0 || pool.pad_bottom < 0 || pool.pad_left < 0 || pool.pad_right < 0 ||
        pool.pad_top >= R || pool.pad_bottom >= R || pool.pad_left >= S || pool.pad_right >= S)
        return fail(QNN_ERR_SHAPE, "pool2d: pads must lie in [0, window size) so every window holds an input cell");
    if ((long long)H + pool.pad_top + pool.pad_bottom < R || (long long)W + pool.pad_left + pool.pad_right < S)
        return fail(QNN_ERR_SHAPE, "pool2d: window larger than the padded input");
    if ((long long)R * S > 65536)
        return fail(QNN_ERR_UNSUPPORTED, "pool2d: windows of more than 65536 cells are not supported");
    const int Ho = (H + pool.pad_top + pool.pad_bottom - R) / pool.stride_h + 1;
    const int Wo = (W + pool.pad_left + pool.pad_right - S) / pool.stride_w + 1;
    if ((long long)N * H * W * C >= (1LL << 31) || (long long)N * Ho * Wo * C >= (1LL << 31))
        return fail(QNN_ERR_UNSUPPORTED, "pool2d: tensors of 2^31 or more elements are not supported");
    if (N == 0)
        return QNN_OK;
    if (!x || !y)
        return fail(QNN_ERR_NULL, "pool2d: x or y is NULL");
    const uintptr_t ax = (uintptr_t)x, ay = (uintptr_t)y;
    int vec = (C % 16 == 0 && ax % 16 == 0 && ay % 16 == 0) ? 16
              : (C % 4 == 0 && ax % 4 == 0 && ay % 4 == 0) ? 4 : 1;
    // few output pixels (global pooling): with windows of 8 or more cells,
    // several waves share each pixel's window; otherwise fewer channels per
    // thread, so that the chip holds enough threads
    const long long pix = (long long)N * Ho * Wo;
    const bool split = pix * (C / vec) < 65536 && R * S >= 8 && pix * ((C + 255) / 256) < (1LL << 31);
    if (split)
        vec = vec >= 4 ? 4 : 1;
    while (!split && vec > 1 && pix * (C / vec) < 65536)
        vec /= 4;
    PoolArgs a{};
    a.x = x;
    a.y = y;
    a.N = N; a.H = H; a.W = W; a.C = C; a.R = R; a.S = S;
    a.sh = pool.stride_h; a.sw = pool.stride_w; a.pt = pool.pad_top; a.pl = pool.pad_left;
    a.Ho = Ho; a.Wo = Wo;
    a.mode = avg ? 0 : 1;
    a.count_pad = avg ? count_pad : 0;
    a.zp = a.count_pad ? zero_point : 0;
    a.rounding = rounding == QNN_ROUND_HALF_AWAY ? 1 : 0;
    const hipError_t e = split ? launch_pool_split(a, sgn, vec, (hipStream_t)stream)
                               : launch_pool(a, sgn, vec, (hipStream_t)stream);
    return e == hipSuccess ? QNN_OK : hip_fail(e, "pool2d launch");
}

// qnn.add parameters: each operand requantized to the output scale,
// summed, zp_y added, clamped to the output dtype and activation.
qnn_status make_add_args(qnn_dtype a_dtype, qnn_qparams a_q, qnn_dtype b_dtype, qnn_qparams b_q, qnn_dtype y_dtype,
                         qnn_qparams y_q, qnn_clamp act, qnn_rounding rounding, AddArgs *out)
{
    if (a_dtype != QNN_UINT8 && a_dtype != QNN_INT8)
        return fail(QNN_ERR_DTYPE, "add: a must be uint8 or int8");
    if (b_dtype != QNN_UINT8 && b_dtype != QNN_INT8)
        return fail(QNN_ERR_DTYPE, "add: b must be uint8 or int8");
    if (y_dtype != QNN_UINT8 && y_dtype != QNN_INT8)
        return fail(QNN_ERR_DTYPE, "add: y must be uint8 or int8");
    if (rounding < QNN_ROUND_HALF_UP || rounding > QNN_ROUND_TWO_STAGE)
        return fail(QNN_ERR_QPARAM, "add: unknown rounding %d", (int)rounding);
    qnn_status s;
    if ((s = check_qparams(a_q, "a qparams", 1, a_dtype, false)) != QNN_OK ||
        (s = check_qparams(b_q, "b qparams", 1, b_dtype, false)) != QNN_OK ||
        (s = check_qparams(y_q, "y qparams", 1, y_dtype, false)) != QNN_OK)
        return s;
    AddArgs args{};
    if ((s = out_bounds(y_dtype, act, &args.lo, &args.hi)) != QNN_OK)
        return s;
    const double Ma = (double)a_q.scale[0] / (double)y_q.scale[0];
    const double Mb = (double)b_q.scale[0] / (double)y_q.scale[0];
    if (!derive_multiplier(Ma, &args.ma, &args.na) || !derive_multiplier(Mb, &args.mb, &args.nb))
        return fail(QNN_ERR_QPARAM, "add: multiplier out of range (%g, %g)", Ma, Mb);
    args.na = std::min(args.na, 63);
    args.nb = std::min(args.nb, 63);
    args.zpa = a_q.zero_point[0];
    args.zpb = b_q.zero_point[0];
    args.zp_y = y_q.zero_point[0];
    args.rounding = rounding;
    // 24-bit product form of the rounding (8-bit operands, ties up, shifts
    // in [17, 40], nonzero multipliers)
    args.fast = rounding == QNN_ROUND_HALF_UP && args.ma > 0 && args.mb > 0 && args.na >= 17 && args.na <= 40 &&
                args.nb >= 17 && args.nb <= 40;
    // A term is round((v - zp) * m / 2^n) with |v - zp| at most that of the
    // dtype's ends, within 2 of the real product: bound the sum of both
    // terms and zp_y to decide whether int32 tables of the terms are exact.
    auto term_bound = [](qnn_dtype dt, int32_t zp, int32_t m, int32_t n) {
        const double lo = dt == QNN_INT8 ? -128.0 : 0.0, hi = dt == QNN_INT8 ? 127.0 : 255.0;
        const double v = std::max(std::fabs(lo - zp), std::fabs(hi - zp));
        return v * (double)m / std::ldexp(1.0, n) + 2.0;
    };
    args.tab_ok = term_bound(a_dtype, args.zpa, args.ma, args.na) + term_bound(b_dtype, args.zpb, args.mb, args.nb) +
                      std::fabs((double)args.zp_y) < std::ldexp(1.0, 30);
    if (args.fast) {
        args.mah = args.ma >> 16;
        args.mal = args.ma & 0xffff;
        args.npa = args.na - 16;
        args.ca = 1 << (args.npa - 1);
        args.mbh = args.mb >> 16;
        args.mbl = args.mb & 0xffff;
        args.npb = args.nb - 16;
        args.cb = 1 << (args.npb - 1);
    }
    *out = args;
    return QNN_OK;
}

qnn_status qnn_add(void *stream, const void *a, qnn_dtype a_dtype, qnn_qparams a_q, const void *b,
                   qnn_dtype b_dtype, qnn_qparams b_q, int64_t count, void *y, qnn_dtype y_dtype,
                   qnn_qparams y_q, qnn_clamp act, qnn_rounding rounding)
{
    AddArgs args{};
    qnn_status s = make_add_args(a_dtype, a_q, b_dtype, b_q, y_dtype, y_q, act, rounding, &args);
    if (s != QNN_OK)
        return s;
    if (count < 0)
        return fail(QNN_ERR_SHAPE, "add: count must be >= 0");
    if (count == 0)
        return QNN_OK;
    if (!a || !b || !y)
        return fail(QNN_ERR_NULL, "add: a, b or y is NULL");
    args.a = a;
    args.b = b;
    args.y = y;
    args.count = count;
    const bool aligned = (((uintptr_t)a | (uintptr_t)b | (uintptr_t)y) & 15) == 0;
    const hipError_t e = launch_add(args, a_dtype, b_dtype, y_dtype, aligned, (hipStream_t)stream);
    return e == hipSuccess ? QNN_OK : hip_fail(e, "add launch");
}

qnn_status qnn_plan_set_residual(qnn_plan *plan, qnn_dtype r_dtype, qnn_qparams r_q, int32_t r_ldc, int32_t r_coff,
                                 qnn_dtype o_dtype, qnn_qparams o_q, qnn_clamp act, qnn_rounding rounding)
{
    if (!plan)
        return fail(QNN_ERR_NULL, "plan_set_residual: plan is NULL");
    if (plan->kind != PLAN_CONV)
        return fail(QNN_ERR_UNSUPPORTED, "plan_set_residual: conv and dense plans only");
    if (plan->fused)
        return fail(QNN_ERR_UNSUPPORTED, "plan_set_residual: the plan already adds a residual");
    const ConvArgs &c = plan->conv;
    const int wave_tile = plan->ker.fam == FAM_DMA   ? dma_wave_tile(plan->ker.tile)
                          : plan->ker.fam == FAM_TAP ? tap_wave_tile(plan->ker.tile)
                                                     : 0;
    if (plan->mode != OUT_REQUANT || !c.staged || wave_tile == 0 || wave_tile > kFuseMaxWaveTile)
        return fail(QNN_ERR_UNSUPPORTED,
                    "plan_set_residual: the plan's kernel has no fused-add epilogue (8-bit output staged by the "
                    "tap-walk or LDS-direct kernels whose waves hold at most 64 x 64 outputs)");
    if (c.ksplit > 1)
        return fail(QNN_ERR_UNSUPPORTED, "plan_set_residual: the plan's kernel splits the reduction (the fused add "
                                         "has no split form)");
    if (c.y_ldc % 16 != 0 || c.y_coff % 16 != 0)
        return fail(QNN_ERR_UNSUPPORTED, "plan_set_residual: the fused add stores 16-byte output rows; y_ldc %d and "
                                         "y_coff %d must be multiples of 16", c.y_ldc, c.y_coff);
    if (r_coff < 0 || r_ldc < (int64_t)r_coff + c.K)
        return fail(QNN_ERR_SHAPE, "plan_set_residual: residual row stride %d and channel offset %d do not hold %d "
                                   "channels", r_ldc, r_coff, c.K);
    if ((int64_t)c.M * r_ldc >= (int64_t(1) << 31))
        return fail(QNN_ERR_UNSUPPORTED, "plan_set_residual: residual of 2^31 bytes or more");
    const float ys = plan->y_scale;
    const int32_t yz = plan->y_zp;
    const qnn_qparams y_q{&ys, &yz, 1};
    AddArgs args{};
    qnn_status s = make_add_args((qnn_dtype)plan->y_dt, y_q, r_dtype, r_q, o_dtype, o_q, act, rounding, &args);
    if (s != QNN_OK)
        return s;
    // term tables (one term per operand byte) where they are exact
    if (args.tab_ok) {
        hipError_t e;
        if ((e = hipMalloc((void **)&plan->addtab, 512 * sizeof(int32_t))) != hipSuccess) {
            plan->addtab = nullptr;
            return fail(QNN_ERR_ALLOC, "plan_set_residual: table allocation: %s", hipGetErrorString(e));
        }
        if ((e = launch_add_table(args, plan->y_dt == QNN_INT8 ? 1 : 0, r_dtype == QNN_INT8 ? 1 : 0, plan->addtab,
                                  nullptr)) != hipSuccess ||
            (e = hipStreamSynchronize(nullptr)) != hipSuccess) {
            (void)hipFree(plan->addtab);
            plan->addtab = nullptr;
            return hip_fail(e, "plan_set_residual: table kernel");
        }
        args.tab = plan->addtab;
    }
    plan->conv.fadd = args;
    plan->conv.r_ldc = r_ldc;
    plan->conv.r_coff = r_coff;
    plan->conv.rdt = r_dtype == QNN_INT8 ? 1 : 0;
    plan->fused = true;
    plan->desc += args.tab ? " +add" : " +add(no-tables)";
    return QNN_OK;
}

qnn_status qnn_plan_run_residual(const qnn_plan *plan, void *stream, const void *x, const void *residual, void *y,
                                 void *workspace)
{
    if (!plan)
        return fail(QNN_ERR_NULL, "plan_run_residual: plan is NULL");
    if (!plan->fused)
        return fail(QNN_ERR_UNSUPPORTED, "plan_run_residual: the plan adds no residual (qnn_plan_set_residual)");
    if (plan->conv.M == 0)
        return QNN_OK;   // empty batch: nothing to read or write, as in qnn_plan_run
    if (!residual)
        return fail(QNN_ERR_NULL, "plan_run_residual: residual is NULL");
    return run_plan(plan, (hipStream_t)stream, x, y, workspace, residual);
}

qnn_status qnn_conv2d_plan_create(qnn_plan **plan, void *stream, qnn_dtype x_dtype, int32_t N, int32_t H,
                                  int32_t W, int32_t C, qnn_qparams x_q, const int8_t *w, int32_t K, int32_t R,
                                  int32_t S, qnn_qparams w_q, const int32_t *bias, qnn_conv_params conv,
                                  qnn_dtype y_dtype, qnn_qparams y_q, qnn_clamp act, qnn_rounding rounding,
                                  int32_t y_ldc, int32_t y_coff)
{
    if (!plan)
        return fail(QNN_ERR_NULL, "plan_create: plan pointer is NULL");
    *plan = nullptr;
    const ConvDesc d = conv_desc(x_dtype, N, H, W, C, x_q, w, K, R, S, w_q, bias, conv, y_dtype, y_q, act,
                                 rounding, y_ldc, y_coff, false);
    qnn_plan *p = nullptr;
    qnn_status s = make_conv_plan(d, (hipStream_t)stream, &p);
    if (s == QNN_OK && (s = alloc_ws(p)) != QNN_OK) {
        free_plan(p);
        return s;
    }
    *plan = p;
    return s;
}

qnn_status qnn_depthwise_conv2d_plan_create(qnn_plan **plan, void *stream, qnn_dtype x_dtype, int32_t N, int32_t H,
                                            int32_t W, int32_t C, qnn_qparams x_q, const int8_t *w, int32_t R,
                                            int32_t S, qnn_qparams w_q, const int32_t *bias, qnn_conv_params conv,
                                            qnn_dtype y_dtype, qnn_qparams y_q, qnn_clamp act,
                                            qnn_rounding rounding, int32_t y_ldc, int32_t y_coff)
{
    if (!plan)
        return fail(QNN_ERR_NULL, "plan_create: plan pointer is NULL");
    *plan = nullptr;
    const ConvDesc d = conv_desc(x_dtype, N, H, W, C, x_q, w, C, R, S, w_q, bias, conv, y_dtype, y_q, act,
                                 rounding, y_ldc, y_coff, true);
    return make_conv_plan(d, (hipStream_t)stream, plan);
}

qnn_status qnn_dense_plan_create(qnn_plan **plan, void *stream, qnn_dtype x_dtype, int32_t M, int32_t Kd,
                                 qnn_qparams x_q, const int8_t *w, int32_t Nd, qnn_qparams w_q, const int32_t *bias,
                                 qnn_dtype y_dtype, qnn_qparams y_q, qnn_clamp act, qnn_rounding rounding,
                                 int32_t y_ldc)
{
    if (!plan)
        return fail(QNN_ERR_NULL, "plan_create: plan pointer is NULL");
    *plan = nullptr;
    if (M < 0)
        return fail(QNN_ERR_SHAPE, "dense: M must be >= 0");
    const ConvDesc d = dense_desc(x_dtype, M, Kd, x_q, w, Nd, w_q, bias, y_dtype, y_q, act, rounding, y_ldc);
    qnn_plan *p = nullptr;
    qnn_status s = make_conv_plan(d, (hipStream_t)stream, &p);
    if (s == QNN_OK && (s = alloc_ws(p)) != QNN_OK) {
        free_plan(p);
        return s;
    }
    *plan = p;
    return s;
}

qnn_status qnn_conv2d_plan_create_wt(qnn_plan **plan, void *stream, qnn_dtype x_dtype, int32_t N, int32_t H,
                                     int32_t W, int32_t C, qnn_qparams x_q, const void *w, qnn_dtype w_dtype,
                                     int32_t K, int32_t R, int32_t S, qnn_qparams w_q, const int32_t *bias,
                                     qnn_conv_params conv, qnn_dtype y_dtype, qnn_qparams y_q, qnn_clamp act,
                                     qnn_rounding rounding, int32_t y_ldc, int32_t y_coff)
{
    if (!plan)
        return fail(QNN_ERR_NULL, "plan_create: plan pointer is NULL");
    *plan = nullptr;
    const size_t n = K > 0 && R > 0 && S > 0 && C > 0 ? (size_t)K * R * S * C : 0;
    LegalWeights lw;
    const int8_t *w8 = nullptr;
    qnn_qparams wq8{};
    qnn_status s = legalize_weights(w, w_dtype, n, w_q, K, (hipStream_t)stream, &lw, &w8, &wq8);
    if (s != QNN_OK)
        return s;
    return qnn_conv2d_plan_create(plan, stream, x_dtype, N, H, W, C, x_q, w8, K, R, S, wq8, bias, conv, y_dtype,
                                  y_q, act, rounding, y_ldc, y_coff);
}

qnn_status qnn_depthwise_conv2d_plan_create_wt(qnn_plan **plan, void *stream, qnn_dtype x_dtype, int32_t N,
                                               int32_t H, int32_t W, int32_t C, qnn_qparams x_q, const void *w,
                                               qnn_dtype w_dtype, int32_t R, int32_t S, qnn_qparams w_q,
                                               const int32_t *bias, qnn_conv_params conv, qnn_dtype y_dtype,
                                               qnn_qparams y_q, qnn_clamp act, qnn_rounding rounding, int32_t y_ldc,
                                               int32_t y_coff)
{
    if (!plan)
        return fail(QNN_ERR_NULL, "plan_create: plan pointer is NULL");
    *plan = nullptr;
    const size_t n = R > 0 && S > 0 && C > 0 ? (size_t)R * S * C : 0;
    LegalWeights lw;
    const int8_t *w8 = nullptr;
    qnn_qparams wq8{};
    qnn_status s = legalize_weights(w, w_dtype, n, w_q, C, (hipStream_t)stream, &lw, &w8, &wq8);
    if (s != QNN_OK)
        return s;
    return qnn_depthwise_conv2d_plan_create(plan, stream, x_dtype, N, H, W, C, x_q, w8, R, S, wq8, bias, conv,
                                            y_dtype, y_q, act, rounding, y_ldc, y_coff);
}

qnn_status qnn_dense_plan_create_wt(qnn_plan **plan, void *stream, qnn_dtype x_dtype, int32_t M, int32_t Kd,
                                    qnn_qparams x_q, const void *w, qnn_dtype w_dtype, int32_t Nd, qnn_qparams w_q,
                                    const int32_t *bias, qnn_dtype y_dtype, qnn_qparams y_q, qnn_clamp act,
                                    qnn_rounding rounding, int32_t y_ldc)
{
    if (!plan)
        return fail(QNN_ERR_NULL, "plan_create: plan pointer is NULL");
    *plan = nullptr;
    const size_t n = Nd > 0 && Kd > 0 ? (size_t)Nd * Kd : 0;
    LegalWeights lw;
    const int8_t *w8 = nullptr;
    qnn_qparams wq8{};
    qnn_status s = legalize_weights(w, w_dtype, n, w_q, Nd, (hipStream_t)stream, &lw, &w8, &wq8);
    if (s != QNN_OK)
        return s;
    return qnn_dense_plan_create(plan, stream, x_dtype, M, Kd, x_q, w8, Nd, wq8, bias, y_dtype, y_q, act, rounding,
                                 y_ldc);
}

qnn_status qnn_requantize_plan_create(qnn_plan **plan, void *stream, qnn_dtype x_dtype, int64_t count,
                                      int32_t channels, qnn_qparams x_q, qnn_dtype y_dtype, qnn_qparams y_q,
                                      qnn_clamp act, qnn_rounding rounding)
{
    if (!plan)
        return fail(QNN_ERR_NULL, "plan_create: plan pointer is NULL");
    *plan = nullptr;
    return make_req_plan(x_dtype, count, channels, x_q, y_dtype, y_q, act, rounding, (hipStream_t)stream, true,
                         plan);
}

qnn_status qnn_plan_run(const qnn_plan *plan, void *stream, const void *x, void *y, void *workspace)
{
    if (!plan)
        return fail(QNN_ERR_NULL, "plan_run: plan is NULL");
    return run_plan(plan, (hipStream_t)stream, x, y, workspace);
}

qnn_status qnn_plan_run_timed(const qnn_plan *plan, void *stream, const void *x, void *y, void *workspace,
                              void *start_event, void *stop_event)
{
    if (!plan)
        return fail(QNN_ERR_NULL, "plan_run_timed: plan is NULL");
    if (!start_event || !stop_event)
        return fail(QNN_ERR_NULL, "plan_run_timed: an event is NULL");
    if (plan->kind != PLAN_CONV && plan->kind != PLAN_DW)
        return fail(QNN_ERR_UNSUPPORTED, "plan_run_timed: conv, dense and depthwise plans only");
    LaunchEvents &ev = launch_events();
    ev.start = (hipEvent_t)start_event;
    ev.stop = (hipEvent_t)stop_event;
    const qnn_status s = run_plan(plan, (hipStream_t)stream, x, y, workspace);
    ev = LaunchEvents{};
    return s;
}

qnn_status qnn_time_next_kernel(void *start_event, void *stop_event)
{
    LaunchEvents &ev = launch_events();
    ev.start = (hipEvent_t)start_event;
    ev.stop = (hipEvent_t)stop_event;
    if (!start_event || !stop_event)
        ev = LaunchEvents{};
    return QNN_OK;
}

qnn_status qnn_plan_run_noalloc(const qnn_plan *plan, void *stream, const void *x, void *y)
{
    if (!plan)
        return fail(QNN_ERR_NULL, "plan_run_noalloc: plan is NULL");
    const size_t data = plan->ws_bytes - plan->ws_cnt_bytes;
    if (plan->ws_cnt_bytes > kScratchCntBytes || data > kScratchBytes - kScratchCntBytes)
        return fail(QNN_ERR_UNSUPPORTED,
                    "plan_run_noalloc: the plan needs %zu bytes of counters and %zu of workspace, the static scratch "
                    "holds %zu and %zu",
                    plan->ws_cnt_bytes, data, kScratchCntBytes, kScratchBytes - kScratchCntBytes);
    if (!plan->ws_bytes)
        return run_plan_at(plan, (hipStream_t)stream, x, y, nullptr, nullptr);
    char *sc = nullptr;
    qnn_status s = scratch_for_device((hipStream_t)stream, &sc);
    if (s != QNN_OK)
        return s;
    return run_plan_at(plan, (hipStream_t)stream, x, y, sc, sc + kScratchCntBytes);
}

size_t qnn_plan_workspace_size(const qnn_plan *plan) { return plan ? plan->ws_bytes : 0; }

const char *qnn_plan_describe(const qnn_plan *plan) { return plan ? plan->desc.c_str() : ""; }

qnn_status qnn_set_tuning_file(const char *path)
{
    std::map<std::string, ConvKernel> rec;
    if (path && *path) {
        FILE *f = std::fopen(path, "r");
        if (!f && errno != ENOENT)
            return fail(QNN_ERR_UNSUPPORTED, "cannot read the tuning file %s: %s", path, std::strerror(errno));
        if (f) {
            char line[512], key[256];
            while (std::fgets(line, sizeof line, f)) {
                int fam = 0, tile = 0, split = 1;
                const int n = std::sscanf(line, "%255s %d %d %d", key, &fam, &tile, &split);
                if (n >= 3 && fam >= FAM_GATHER && fam <= FAM_WIN && tile >= 0 && split >= 1)
                    rec[key] = ConvKernel{fam, tile, n == 4 ? split : 1};
            }
            std::fclose(f);
        }
    }
    std::lock_guard<std::mutex> g(g_tune_mu);
    g_tune.swap(rec);
    g_tune_path = path ? path : "";
    return QNN_OK;
}

void qnn_plan_destroy(qnn_plan *plan) { free_plan(plan); }

}  // extern "C"
