/*
 * qnn.h -- C ABI of libqnn: quantized (INT8) conv2d, depthwise conv2d and
 * dense fused with requantize, plus standalone requantize and add, for AMD
 * Instinct MI355X (gfx950).
 *
 * Problem statement (Jain et al., "Efficient Execution of Quantized Deep
 * Learning Models: A Compiler Approach"):
 *   - Sec. I-A, Eq. (1): a quantized tensor is Q plus (scale, zero_point) and
 *     stands for the real tensor scale * (Q - zero_point).  Scales may be per
 *     tensor or, for weights, per output channel; zero points make the
 *     quantization asymmetric (Sec. II-A, Table I lists asymmetric,
 *     symmetric and per-channel quantization).
 *   - Sec. II-B, Eq. (2)/(3): the quantized conv2d output is the int32
 *     accumulator sum_{c,r,s} (Q_A - zp_A)(Q_B - zp_B) with scale
 *     scale_A * scale_B and zero point 0; Eq. (3) splits it into four terms.
 *   - Sec. III-B: padding uses the input zero point; requantize (Eq. (5))
 *     maps a quantized tensor to another (scale, zero_point) with a
 *     fixed-point multiplier; the rounding is a choice (three are offered).
 *   - Sec. III-A, Fig. 2: a framework conv is qnn.conv2d -> bias_add -> clip
 *     -> requantize; here the clip is applied in the output Q domain after
 *     requantize (identical for ReLU).
 *
 * Conventions for every entry point:
 *   - Tensor data (x, w, bias, y) are DEVICE pointers owned by the caller;
 *     the library never frees them.  Quantization attributes (scale and zero
 *     point arrays inside qnn_qparams) are HOST arrays read during the call.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Work is enqueued on it; one-shot calls synchronize it before they
 *     return (they upload per-channel tables), plan runs do not.
 *   - Layouts: activations NHWC; conv weights OHWI, i.e. [K][R][S][C] with C
 *     fastest; depthwise weights [R][S][C]; dense x [M][Kd], w [Nd][Kd];
 *     outputs NHWC / [M][Nd] with a row stride y_ldc (elements) and a
 *     channel offset y_coff, so a branch can write its slice of a concat.
 *   - Every function returns a qnn_status; on failure nothing is enqueued
 *     and qnn_last_error() describes the problem.  There are no aborts and
 *     no exceptions across the ABI.  Asynchronous device faults surface at
 *     the caller's next synchronization.
 *   - Validation (before any device work): scales finite and > 0 (a weight
 *     scale of exactly 0 is allowed and yields zp_out); zero points inside
 *     the range of their dtype (weights: int8); output clamp non-empty after
 *     intersection with the output dtype range; the requantize multiplier
 *     s_x*s_w[k]/s_y must have a fixed-point shift >= 1 (M below about
 *     2^30); the integer accumulator must provably fit int32:
 *     J * max|x - zp_x| * max|w - zp_w[k]| + |bias[k]| < 2^31 with
 *     J = R*S*C, else QNN_ERR_OVERFLOW; input and output tensors below 2^31
 *     elements.  Empty inputs (N == 0, M == 0, count == 0) are valid no-ops.
 */
#ifndef QNN_H
#define QNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define QNN_ABI_VERSION 1

/* The enums are int-sized in C.  In C++ they get int as their fixed
 * underlying type, so that every int a caller passes is a value of the
 * enum type (the library validates it) rather than an out-of-range one. */
#ifdef __cplusplus
#define QNN_ENUM_INT : int
#else
#define QNN_ENUM_INT
#endif

typedef enum QNN_ENUM_INT {
    QNN_OK = 0,
    QNN_ERR_NULL = 1,        /* a required pointer is NULL */
    QNN_ERR_SHAPE = 2,       /* non-positive or inconsistent sizes, bad y_ldc/y_coff */
    QNN_ERR_DTYPE = 3,       /* dtype not allowed for this argument */
    QNN_ERR_QPARAM = 4,      /* bad scale / zero point / clamp / multiplier */
    QNN_ERR_OVERFLOW = 5,    /* int32 accumulator bound cannot be guaranteed */
    QNN_ERR_UNSUPPORTED = 6, /* valid but not supported (e.g. too large) */
    QNN_ERR_HIP = 7,         /* a HIP runtime call or kernel launch failed */
    QNN_ERR_ALLOC = 8        /* device or host allocation failed */
} qnn_status;

typedef enum QNN_ENUM_INT { QNN_UINT8 = 0, QNN_INT8 = 1, QNN_INT32 = 2 } qnn_dtype;

/* Rounding of the fixed-point requantize (the paper leaves it to the
 * framework, Sec. III-B): HALF_UP rounds round(v * mult / 2^shift) with ties
 * toward +infinity, HALF_AWAY with ties away from zero.  TWO_STAGE is the
 * integer-only form of Jacob et al. used by pre-quantized TFLite models:
 * for shift >= 31 the product is divided by 2^31 rounding half up, and that
 * integer by 2^(shift - 31) rounding half away from zero (two roundings,
 * so a result may differ by 1 from either single rounding); for shift < 31
 * (multipliers of 1 or more) one half-up rounding. */
typedef enum QNN_ENUM_INT { QNN_ROUND_HALF_UP = 0, QNN_ROUND_HALF_AWAY = 1, QNN_ROUND_TWO_STAGE = 2 } qnn_rounding;

/* Quantization attributes of one tensor (host arrays).  n == 1: per tensor;
 * n == channel count: per output channel (weights) or per innermost channel
 * (standalone requantize). */
typedef struct {
    const float *scale;
    const int32_t *zero_point;
    int32_t n;
} qnn_qparams;

typedef struct {
    int32_t stride_h, stride_w;
    int32_t pad_top, pad_left, pad_bottom, pad_right;
    int32_t dil_h, dil_w;
} qnn_conv_params;

/* Activation clamp in the OUTPUT Q domain, intersected with the output
 * dtype range.  No clamp: {INT32_MIN, INT32_MAX}; ReLU: {zp_out, INT32_MAX}. */
typedef struct {
    int32_t lo, hi;
} qnn_clamp;

typedef struct qnn_plan qnn_plan;

/* ---------------------------------------------------------------- info */

int32_t qnn_abi_version(void);

/* Thread-local message for the last non-OK status returned on this thread. */
const char *qnn_last_error(void);

const char *qnn_status_string(qnn_status s);

/*
 * Fixed-point form of a real multiplier (Sec. III-B, Eq. (5)): M >= 0 is
 * written M = f * 2^e with f in [0.5, 1); mult = floor(f * 2^31 + 1/2),
 * renormalised to 2^30 (e + 1) when it reaches 2^31; shift = 31 - e.  On
 * success mult is in [2^30, 2^31) and shift >= 1 (shift may exceed 63, in
 * which case every product rounds to 0); M == 0 gives mult 0, shift 1.
 * Returns QNN_ERR_QPARAM for negative, non-finite or too large M.  Pure host
 * function, no device work.
 */
qnn_status qnn_quantize_multiplier(double M, int32_t *mult, int32_t *shift);

/* ---------------------------------------------------------------- conv2d */

/*
 * qnn.conv2d + bias + requantize + clamp (Eq. (2)/(3) and (5); Fig. 2).
 *   x: device, x_dtype UINT8 or INT8, NHWC [N][H][W][C]; x_q per tensor.
 *   w: device, int8 OHWI [K][R][S][C]; w_q per tensor or per channel (n == K),
 *      weight zero points in [-128, 127].
 *   bias: device int32 [K] with implied scale s_x*s_w[k] and zero point 0,
 *      or NULL.
 *   conv: strides >= 1, pads >= 0, dilations >= 1; padded taps hold zp_x.
 *   y: device, NHWC with Ho = (H + pt + pb - dil_h*(R-1) - 1)/stride_h + 1
 *      (same for Wo); element (m, k), m = (n*Ho + oh)*Wo + ow, is stored at
 *      y[m*y_ldc + y_coff + k]; y_ldc >= y_coff + K, y_coff >= 0.
 *      y_dtype UINT8 / INT8: requantized with y_q (per tensor), clamp `act`
 *      and `rounding`.  y_dtype INT32: the raw accumulator plus bias (the
 *      qnn.conv2d output of Eq. (2)); y_q, act and rounding are ignored.
 * Synchronizes `stream` before returning.
 */
qnn_status qnn_conv2d(void *stream,
                      const void *x, qnn_dtype x_dtype, int32_t N, int32_t H, int32_t W,
                      int32_t C, qnn_qparams x_q,
                      const int8_t *w, int32_t K, int32_t R, int32_t S, qnn_qparams w_q,
                      const int32_t *bias, qnn_conv_params conv,
                      void *y, qnn_dtype y_dtype, qnn_qparams y_q, qnn_clamp act,
                      qnn_rounding rounding, int32_t y_ldc, int32_t y_coff);

/*
 * Depthwise conv2d with channel multiplier 1 + bias + requantize + clamp:
 * acc[n,oh,ow,c] = sum_{r,s} (x~[.., c] - zp_x)(w[r][s][c] - zp_w[c]) + bias[c].
 * This is Eq. (2) with each output channel reading only its own input
 * channel (so J = R*S), evaluated in the subtract-first form that Sec.
 * III-B gives as the alternative lowering of the QNN convolution; x~ is x
 * inside the image and zp_x in the padding (Sec. III-B); the requantize is
 * Eq. (5).
 *   w: device int8 [R][S][C]; w_q per tensor or per channel (n == C).
 *   y: NHWC [N][Ho][Wo][C] with row stride y_ldc >= y_coff + C.
 * Other arguments as qnn_conv2d.  Synchronizes `stream` before returning.
 */
qnn_status qnn_depthwise_conv2d(void *stream,
                                const void *x, qnn_dtype x_dtype, int32_t N, int32_t H,
                                int32_t W, int32_t C, qnn_qparams x_q,
                                const int8_t *w, int32_t R, int32_t S, qnn_qparams w_q,
                                const int32_t *bias, qnn_conv_params conv,
                                void *y, qnn_dtype y_dtype, qnn_qparams y_q, qnn_clamp act,
                                qnn_rounding rounding, int32_t y_ldc, int32_t y_coff);

/*
 * qnn.dense + bias + requantize + clamp:
 * acc[m,j] = sum_k (x[m,k] - zp_x)(w[j,k] - zp_w[j]) + bias[j].
 * Sec. III-D names matrix multiplication beside conv2d as the operators
 * whose integer schedules need data reuse; its accumulator is Eq. (2)/(3)
 * with a 1x1 window over Kd input channels (the four terms of Eq. (3) with
 * J = Kd), followed by the requantize of Eq. (5).
 *   x: device [M][Kd] (UINT8/INT8), w: device int8 [Nd][Kd], bias [Nd] or NULL,
 *   y: device [M][y_ldc] with y_ldc >= Nd.  Synchronizes `stream`.
 */
qnn_status qnn_dense(void *stream,
                     const void *x, qnn_dtype x_dtype, int32_t M, int32_t Kd, qnn_qparams x_q,
                     const int8_t *w, int32_t Nd, qnn_qparams w_q, const int32_t *bias,
                     void *y, qnn_dtype y_dtype, qnn_qparams y_q, qnn_clamp act,
                     qnn_rounding rounding, int32_t y_ldc);

/* ---------------------------------------------------------------- elementwise */

/*
 * Standalone requantize (Eq. (5)):
 *   y[i] = clamp(zp_out[c] + round((x[i] - zp_in[c]) * s_in[c] / s_out[c]))
 * with c = i % channels (innermost axis); x_q and y_q per tensor (n == 1)
 * or per channel (n == channels).  x_dtype UINT8, INT8 or INT32 (INT32
 * requires zero point 0, the qnn.conv2d output convention of Eq. (2));
 * y_dtype UINT8, INT8 or INT32.  x and y are device arrays of `count`
 * elements and must not overlap.  Enqueued on `stream`; synchronizes it
 * only when per-channel parameters are uploaded.
 */
qnn_status qnn_requantize(void *stream, const void *x, qnn_dtype x_dtype, int64_t count,
                          int32_t channels, qnn_qparams x_q,
                          void *y, qnn_dtype y_dtype, qnn_qparams y_q, qnn_clamp act,
                          qnn_rounding rounding);

/*
 * qnn.add of two same-shape tensors with different per-tensor qparams:
 *   y = clamp(zp_y + round((a - zp_a) * s_a / s_y) + round((b - zp_b) * s_b / s_y))
 * A quantized add is named among the operators a framework adds (Sec. I-B)
 * but its lowering is not given; this follows the paper's principle that a
 * quantized operator decomposes into simpler existing ones (Sec. II-B, and
 * Sec. III-A: QNN operators are wrappers around sequences of them): each
 * input is requantized to the output scale by Eq. (5) without its zero
 * point, the two integers are added, then zp_y is added and the result
 * clamped.
 * a, b: device UINT8/INT8 arrays of `count` elements; y: UINT8/INT8.
 * Enqueued on `stream`, no synchronization.
 */
qnn_status qnn_add(void *stream, const void *a, qnn_dtype a_dtype, qnn_qparams a_q,
                   const void *b, qnn_dtype b_dtype, qnn_qparams b_q, int64_t count,
                   void *y, qnn_dtype y_dtype, qnn_qparams y_q, qnn_clamp act,
                   qnn_rounding rounding);

typedef enum QNN_ENUM_INT {
    QNN_POOL_AVG = 0,
    QNN_POOL_MAX = 1
} qnn_pool_mode;

/*
 * Quantized 2-D pooling, Eq. (4) (Sec. III-B, QNN pooling): input and output
 * share one scale and zero point, so the quantized output is the pooled
 * quantized input and no scale is involved.
 *   x: device NHWC [N][H][W][C], UINT8 or INT8; y: device NHWC
 *      [N][Ho][Wo][C] of the same dtype, Ho = (H + pad_top + pad_bottom -
 *      R)/stride_h + 1, Wo likewise.
 *   pool: strides >= 1, dilations 1, pads with 0 <= pad_top, pad_bottom < R
 *      and 0 <= pad_left, pad_right < S (so that every window holds a cell
 *      of the input); R*S <= 65536.
 *   mode QNN_POOL_AVG: y = the window sum (exact, int32) divided by its cell
 *      count, rounded to nearest with ties by `rounding` (HALF_UP or
 *      HALF_AWAY; TWO_STAGE is rejected).  count_pad 0 leaves padded cells
 *      out of sum and count; count_pad 1 counts them as holding zero_point
 *      (a real zero), which must then lie in the dtype's range.
 *   mode QNN_POOL_MAX: y = the largest cell of the window inside the input;
 *      count_pad, zero_point and rounding are ignored.
 * N may be 0 (then x and y may be NULL).  Tensors of 2^31 or more elements
 * return QNN_ERR_UNSUPPORTED.  Enqueued on `stream`, no synchronization.
 */
qnn_status qnn_pool2d(void *stream, const void *x, qnn_dtype dtype, int32_t N, int32_t H,
                      int32_t W, int32_t C, int32_t R, int32_t S, qnn_conv_params pool,
                      qnn_pool_mode mode, int32_t count_pad, int32_t zero_point, void *y,
                      qnn_rounding rounding);

/* ---------------------------------------------------------------- plans */

/*
 * Prepared forms.  Weights, bias and quantization parameters are constants
 * of inference (Sec. III-B: terms 2 and 4 of Eq. (3) are compile-time
 * constants and are folded), so a plan reads the weights and bias once,
 * derives the per-channel fixed-point multipliers and the folded constant
 * bias[k] - zp_x*sum_j w[k,j] + J*zp_x*zp_w[k], and packs the weights into
 * device memory it owns.  Arguments mean what they mean in the one-shot
 * calls; x and y are given at run time.  Creation synchronizes `stream`;
 * conv and dense creation also times the candidate kernels on `stream`
 * (see qnn_set_tuning_file), using scratch device memory it frees again.
 * A plan is immutable after creation: runs on different streams may overlap
 * provided each passes its own workspace (see qnn_plan_workspace_size).
 */
qnn_status qnn_conv2d_plan_create(qnn_plan **plan, void *stream,
                                  qnn_dtype x_dtype, int32_t N, int32_t H, int32_t W,
                                  int32_t C, qnn_qparams x_q,
                                  const int8_t *w, int32_t K, int32_t R, int32_t S,
                                  qnn_qparams w_q, const int32_t *bias, qnn_conv_params conv,
                                  qnn_dtype y_dtype, qnn_qparams y_q, qnn_clamp act,
                                  qnn_rounding rounding, int32_t y_ldc, int32_t y_coff);

qnn_status qnn_depthwise_conv2d_plan_create(qnn_plan **plan, void *stream,
                                            qnn_dtype x_dtype, int32_t N, int32_t H,
                                            int32_t W, int32_t C, qnn_qparams x_q,
                                            const int8_t *w, int32_t R, int32_t S,
                                            qnn_qparams w_q, const int32_t *bias,
                                            qnn_conv_params conv, qnn_dtype y_dtype,
                                            qnn_qparams y_q, qnn_clamp act,
                                            qnn_rounding rounding, int32_t y_ldc,
                                            int32_t y_coff);

qnn_status qnn_dense_plan_create(qnn_plan **plan, void *stream,
                                 qnn_dtype x_dtype, int32_t M, int32_t Kd, qnn_qparams x_q,
                                 const int8_t *w, int32_t Nd, qnn_qparams w_q,
                                 const int32_t *bias, qnn_dtype y_dtype, qnn_qparams y_q,
                                 qnn_clamp act, qnn_rounding rounding, int32_t y_ldc);

/*
 * The same three plans for weights given as int8 or asymmetric uint8
 * (w_dtype QNN_INT8 or QNN_UINT8; with uint8 the weight zero points lie in
 * [0, 255]).  Pre-quantized models of some frameworks carry uint8 weights;
 * as Sec. III-C legalises a dtype the instructions do not take (there the
 * activations of Intel's uint8 x int8 dot products), uint8 weights are
 * legalised once at creation: w' = w - 128 read as int8, zp_w' = zp_w - 128,
 * which leaves every (w - zp_w) of Eq. (3), hence every output, unchanged.
 * Everything else as in the plain creation calls; other dtypes return
 * QNN_ERR_DTYPE.
 */
qnn_status qnn_conv2d_plan_create_wt(qnn_plan **plan, void *stream,
                                     qnn_dtype x_dtype, int32_t N, int32_t H, int32_t W,
                                     int32_t C, qnn_qparams x_q,
                                     const void *w, qnn_dtype w_dtype, int32_t K, int32_t R,
                                     int32_t S, qnn_qparams w_q, const int32_t *bias,
                                     qnn_conv_params conv, qnn_dtype y_dtype, qnn_qparams y_q,
                                     qnn_clamp act, qnn_rounding rounding, int32_t y_ldc,
                                     int32_t y_coff);

qnn_status qnn_depthwise_conv2d_plan_create_wt(qnn_plan **plan, void *stream,
                                               qnn_dtype x_dtype, int32_t N, int32_t H,
                                               int32_t W, int32_t C, qnn_qparams x_q,
                                               const void *w, qnn_dtype w_dtype, int32_t R,
                                               int32_t S, qnn_qparams w_q, const int32_t *bias,
                                               qnn_conv_params conv, qnn_dtype y_dtype,
                                               qnn_qparams y_q, qnn_clamp act,
                                               qnn_rounding rounding, int32_t y_ldc,
                                               int32_t y_coff);

qnn_status qnn_dense_plan_create_wt(qnn_plan **plan, void *stream,
                                    qnn_dtype x_dtype, int32_t M, int32_t Kd, qnn_qparams x_q,
                                    const void *w, qnn_dtype w_dtype, int32_t Nd,
                                    qnn_qparams w_q, const int32_t *bias, qnn_dtype y_dtype,
                                    qnn_qparams y_q, qnn_clamp act, qnn_rounding rounding,
                                    int32_t y_ldc);

/* Per-channel standalone requantize prepared once (count fixed). */
qnn_status qnn_requantize_plan_create(qnn_plan **plan, void *stream,
                                      qnn_dtype x_dtype, int64_t count, int32_t channels,
                                      qnn_qparams x_q, qnn_dtype y_dtype, qnn_qparams y_q,
                                      qnn_clamp act, qnn_rounding rounding);

/*
 * Run a plan on `stream`: x and y are device pointers with the shapes given
 * at creation.  `workspace` is a device buffer of at least
 * qnn_plan_workspace_size(plan) bytes, or NULL to use the plan's own
 * workspace (then overlapping runs of the same plan race).  Does not
 * synchronize.
 */
qnn_status qnn_plan_run(const qnn_plan *plan, void *stream, const void *x, void *y,
                        void *workspace);

/*
 * qnn_plan_run for measurement: the plan's main kernel (the conv, dense or
 * depthwise kernel, not the auxiliary window-sum or padding kernels) is
 * launched with hipExtLaunchKernel, which records start_event and
 * stop_event (hipEvent_t, created by the caller, passed as void*) at that
 * kernel's own start and end, so their elapsed time is the kernel's
 * duration as a profiler reports it.  Nothing is recorded when the plan has
 * no output pixels.  Requantize plans return QNN_ERR_UNSUPPORTED.
 */
qnn_status qnn_plan_run_timed(const qnn_plan *plan, void *stream, const void *x, void *y, void *workspace,
                              void *start_event, void *stop_event);

/*
 * For measurement of the one-shot calls (qnn_add, qnn_requantize,
 * qnn_pool2d, ...): the next main kernel that this host thread launches
 * through an entry point records start_event and stop_event (hipEvent_t as
 * void*) at its own start and end, as qnn_plan_run_timed does.  NULL for
 * either event cancels a pending request.  Always returns QNN_OK.
 */
qnn_status qnn_time_next_kernel(void *start_event, void *stop_event);

/*
 * Residual add fused into a conv or dense plan's epilogue.  The paper
 * lowers QNN operators to sequences of simpler ones and relies on operator
 * fusion to run them together (Sec. III-A, III-B); here the qnn.add that
 * follows a conv in a residual block (qnn_add above) runs inside the conv
 * kernel instead of as a pass of its own.  After the call the plan stores
 *   y = qnn_add(c, r)
 * where c is the conv output exactly as the plan computed it (y_dtype,
 * y_q, act, rounding of the plan: the intermediate, never written) and r
 * is a residual of r_dtype (UINT8 / INT8) with per-tensor r_q, element
 * (pixel m, channel k) at r[m * r_ldc + r_coff + k]; the sum has o_dtype
 * (UINT8 / INT8), o_q (per tensor), clamp `act` and `rounding` (those of
 * qnn_add), and is stored where the plan stores its output (y_ldc,
 * y_coff).  The bytes equal those of qnn_plan_run followed by qnn_add.
 * Only plans whose kernel has the fused epilogue (8-bit output staged
 * through LDS by the tap-walk or LDS-direct kernels, qnn_plan_describe
 * starting with "conv_tap" or "conv_dma", with waves of at most 64 x 64
 * outputs and no split reduction) and whose y_ldc and y_coff are
 * multiples of 16 accept it;
 * others, int32 outputs and a second call return QNN_ERR_UNSUPPORTED and
 * leave the plan as it was.  r_ldc >= r_coff + K.  A fused plan runs only
 * through qnn_plan_run_residual.  Where the add's per-byte terms fit 32-bit
 * sums, the call tabulates them in a 2 KB device buffer that the plan owns
 * (allocated here, one small kernel launched on the null stream and
 * waited for); QNN_ERR_ALLOC or QNN_ERR_HIP if that fails, the plan as it
 * was.
 */
qnn_status qnn_plan_set_residual(qnn_plan *plan, qnn_dtype r_dtype, qnn_qparams r_q, int32_t r_ldc,
                                 int32_t r_coff, qnn_dtype o_dtype, qnn_qparams o_q, qnn_clamp act,
                                 qnn_rounding rounding);

/*
 * Runs a plan with a fused residual add: as qnn_plan_run, with the
 * residual device buffer (layout set by qnn_plan_set_residual, not
 * overlapping y).  y must be 16-byte aligned (QNN_ERR_UNSUPPORTED, nothing
 * enqueued).  Enqueued on `stream`, no synchronization.
 */
qnn_status qnn_plan_run_residual(const qnn_plan *plan, void *stream, const void *x, const void *residual, void *y,
                                 void *workspace);

/*
 * Allocation-free run, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): runs the plan like qnn_plan_run, with its workspace taken from
 * a static device array of the library (64 MiB per device: 1 MiB of
 * counters, 63 MiB for the rest), held by each GPU the library runs on
 * until the process ends.  x and y are the caller's device buffers as in
 * qnn_plan_run.  Allocates nothing and does not synchronize; the first
 * call on a device also clears the counter region with a kernel on
 * `stream` and must not be under stream capture (QNN_ERR_UNSUPPORTED).
 * A plan whose workspace exceeds the array returns QNN_ERR_UNSUPPORTED
 * with nothing enqueued.  Every call on one device shares the array:
 * calls that overlap on one GPU (two streams, two threads) race, so such
 * callers must order them or use qnn_plan_run with separate workspaces.
 */
qnn_status qnn_plan_run_noalloc(const qnn_plan *plan, void *stream, const void *x, void *y);

/* Bytes of device workspace a run needs (0 if none).  When the plan uses a
 * split reduction its workspace starts with arrival counters, which must be
 * zero before the first run with that workspace; every run leaves them
 * zero (the plan's own workspace is zeroed at allocation). */
size_t qnn_plan_workspace_size(const qnn_plan *plan);

/* Human-readable kernel choice of the plan, e.g. "conv_dma tile=128x128x64
 * threads=256 stages=4 ..."; valid until the plan is destroyed. */
const char *qnn_plan_describe(const qnn_plan *plan);

/*
 * Kernel-choice file.  A conv or dense plan picks its kernel by timing the
 * eligible candidate kernels on its own shape at creation (each candidate
 * computes the same bytes; only the time differs).  After this call with a
 * path, creation first looks its shape up in the file's records and, when
 * the recorded choice is still a candidate, takes it without timing; a
 * choice it does time is appended to the file as one text line,
 * "<shape key> <family> <config>".  A missing file starts empty.  NULL or
 * "" stops reading and writing any file and forgets the records.  Returns
 * QNN_ERR_UNSUPPORTED when the file exists but cannot be read.  Plans
 * created concurrently with this call see either the old or the new
 * records.
 */
qnn_status qnn_set_tuning_file(const char *path);

/* Frees the plan's device memory (after synchronizing the device). NULL is
 * a no-op. */
void qnn_plan_destroy(qnn_plan *plan);

#ifdef __cplusplus
}
#endif

#endif /* QNN_H */
