// Internal declarations shared by the host side of libqnn (qnn_api.cpp) and
// its HIP kernels.  Not part of the public ABI.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qnn {

// Events that the next main kernel this host thread launches records at its
// own start and end (qnn_plan_run_timed, qnn_time_next_kernel), null when
// nothing is measured.
struct LaunchEvents {
    hipEvent_t start = nullptr, stop = nullptr;
};
LaunchEvents &launch_events();

// Launch of an operator's main kernel (conv, dense, depthwise, requantize,
// add, pool): with timing events set, through hipExtLaunchKernel, which
// records them at the kernel's own start and end (the dispatch itself, as
// the profiler times it) and consumes them; else a plain launch.
template <typename K, typename... A>
inline void launch_main(K kernel, dim3 grid, dim3 block, uint32_t lds, hipStream_t st, A... args)
{
    LaunchEvents &ev = launch_events();
    if (ev.start) {
        hipExtLaunchKernelGGL(kernel, grid, block, lds, st, ev.start, ev.stop, 0, args...);
        ev = LaunchEvents{};
    } else {
        kernel<<<grid, block, lds, st>>>(args...);
    }
}

// Per-output-channel epilogue record of a conv / dense plan.
//   mult   : fixed-point requantize multiplier (Q31 significand)
//   bconst : bias[k] - zp_x' * sum_j w[k,j] + J * zp_x' * zp_w[k]
//            (terms 2 and 4 of Eq. (3) folded with the bias; int32
//            wrap-around arithmetic, exact whenever the true result fits
//            int32, which plan creation guarantees)
//   rndzp  : 32-bit requantize constant 2^(sh-1) + (zp_y + off) * 2^sh with
//            sh = shift - 32 and off = 128 for int8 outputs (0 for uint8);
//            only meaningful when the plan uses the 32-bit requantize
//   shift  : fixed-point shift (clamped to <= 63: every product with a
//            larger shift rounds to 0 anyway)
struct ChanRec {
    int32_t mult, bconst, rndzp, shift;
};

enum OutMode { OUT_REQUANT = 0, OUT_INT32 = 1 };

// Fixed-point requantize of v: round(v * mult / 2^shift) with a 64-bit
// product (|v| <= 2^31, 0 <= mult < 2^31, 1 <= shift <= 63); the mode is the
// public qnn_rounding value.
//   0 HALF_UP: floor((p + 2^(shift-1)) / 2^shift), ties toward +infinity;
//   1 HALF_AWAY: one less is added for negative products, ties away from 0;
//   2 TWO_STAGE (shift >= 31): a rounding high multiply, x1 = floor((p +
//     2^30) / 2^31) (ties up), then x1 / 2^(shift - 31) rounded with ties
//     away from zero (one less added for negative x1), so a product may be
//     rounded twice; for shift < 31 (multipliers of 1 or more) one rounding,
//     as HALF_UP.
// Both code shapes compute the same value; which one leaves a kernel fewer
// registers (and so more resident waves) depends on the kernel: the
// elementwise kernels take the early HALF_UP return (EARLY = true), the
// conv epilogues the single shared rounding.
template <bool EARLY = false>
__device__ __forceinline__ long long rounding_mul_shift(int v, int mult, int shift, int mode)
{
    long long p = (long long)v * (long long)mult;
    if constexpr (EARLY) {
        if (mode == 0)
            return (p + (1LL << (shift - 1))) >> shift;
    }
    if (mode == 2) {
        if (shift > 31) {
            p = (p + (1LL << 30)) >> 31;   // stage 1: / 2^31, ties up
            shift -= 31;                   // stage 2 below: ties away from zero
            mode = 1;
        } else {
            mode = 0;                      // one rounding, ties up
        }
    }
    return (p + (1LL << (shift - 1)) - (mode == 1 && p < 0 ? 1 : 0)) >> shift;
}

// min(max(t, lo), hi) for lo <= hi (the host rejects empty clamps) in one
// VALU operation; the compiler emits a max and a min for runtime bounds.
__device__ __forceinline__ int clamp_i32(int t, int lo, int hi)
{
    int r;
    asm("v_med3_i32 %0, %1, %2, %3" : "=v"(r) : "v"(t), "v"(lo), "v"(hi));
    return r;
}

__device__ __forceinline__ int clampll(long long v, int lo, int hi)
{
    return (int)(v < lo ? lo : (v > hi ? hi : v));
}

// qnn.add arguments (the standalone add kernel, and the residual add fused
// into a conv epilogue).
struct AddArgs {
    const void *a;
    const void *b;
    void *y;
    int64_t count;
    int32_t ma, na, zpa, mb, nb, zpb, zp_y;
    int32_t lo, hi, rounding;
    // HALF_UP with both shifts in [17, 40]: each operand's rounding from two
    // 24-bit products (multiplier halves mh = mult >> 16, ml = mult & 0xffff,
    // np = shift - 16, c = 2^(np - 1)); the operands are 8-bit, so the
    // zero-point-adjusted values fit 9 bits
    int32_t fast, mah, mal, npa, ca, mbh, mbl, npb, cb;
    // tab_ok: every term, and so every sum of two terms plus zp_y, fits 32
    // bits, so that the terms may be tabulated per operand byte as int32
    // (the standalone kernel builds such tables in LDS per workgroup)
    int32_t tab_ok;
    // fused residual add only: tab[b] = add_term_a of the byte b read as
    // the conv output's dtype, tab[256 + b] = add_term_b of the byte b read
    // as the residual's dtype, plus zp_y (512 int32 in device memory, built
    // by add_table_kernel), so that an element's sum is clamp(tab[x] +
    // tab[256 + r]); nullptr where a 32-bit sum could overflow
    const int32_t *tab;
};

// round(v * mult / 2^shift), ties up, for |v| < 2^9 and shift = np + 16 with
// np in [1, 24], from full-rate 24-bit multiplies: p = v * mult = p1 * 2^16 +
// p0 with p1 = v * mh and p0 = v * ml (both exact in 32 bits), so that
// p + 2^(shift-1) = (p1 + c + floor(p0 / 2^16)) * 2^16 + (p0 mod 2^16), and
// the remainder below 2^16 cannot change the floor of the division by
// 2^shift.
__device__ __forceinline__ int round_mul_shift_small(int v, int mh, int ml, int np, int c)
{
    return (__mul24(v, mh) + c + (__mul24(v, ml) >> 16)) >> np;
}

// The two terms of qnn.add: each operand requantized to the output scale,
// round((x - zp_a) * Ma) and round((y - zp_b) * Mb).
__device__ __forceinline__ long long add_term_a(const AddArgs &a, int x)
{
    if (a.fast)
        return round_mul_shift_small(x - a.zpa, a.mah, a.mal, a.npa, a.ca);
    return rounding_mul_shift<true>(x - a.zpa, a.ma, a.na, a.rounding);
}
__device__ __forceinline__ long long add_term_b(const AddArgs &a, int y)
{
    if (a.fast)
        return round_mul_shift_small(y - a.zpb, a.mbh, a.mbl, a.npb, a.cb);
    return rounding_mul_shift<true>(y - a.zpb, a.mb, a.nb, a.rounding);
}

// One element of qnn.add: the two terms summed, zp_y added, clamped (the
// 24-bit form in 32-bit arithmetic, whose terms fit 2^24).
__device__ __forceinline__ int add_one(const AddArgs &a, int x, int y)
{
    if (a.fast)
        return clamp_i32((int)add_term_a(a, x) + (int)add_term_b(a, y) + a.zp_y, a.lo, a.hi);
    return clampll(add_term_a(a, x) + add_term_b(a, y) + a.zp_y, a.lo, a.hi);
}

// Largest wave tile (channels x pixels of one wave) whose epilogue holds
// the fused residual add: waves with larger tiles keep their accumulators
// in most of the register file, and the extra code would spill to
// scratch, whose memory operations share the vector-memory counter that
// the stage waits of the LDS-direct kernels count.
constexpr int kFuseMaxWaveTile = 64 * 64;

// Implicit-GEMM conv arguments.  GEMM view: D[k][m] = sum_j Wp[k][j] * X'[m][j]
// with m = output pixel, k = output channel, j = (r*S + s)*C + c.
struct ConvArgs {
    const uint8_t *x;       // NHWC activations (uint8 or int8 bytes)
    const int8_t *wp;       // packed weights [Kpad][Jpad], zero padded
    const int8_t *wf;       // the same weights in MFMA operand order (conv_wave.hip)
    const ChanRec *chan;    // [Kpad]
    const int32_t *zpw;     // [Kpad] weight zero points (term 3)
    const int32_t *asum;    // [M] window sums of x' (term 3) or nullptr
    const uint8_t *padbuf;  // 16 bytes of zp_x: source of padded / unused gathers
    void *y;                // output (requantized bytes or int32)
    int32_t N, H, W, C, Ho, Wo, R, S;
    int32_t sh, sw, pt, pl, dh, dw;
    int32_t K, Kpad, J, Jpad, M;  // Kpad, Jpad: packed weight rows / row stride
    uint32_t flip4;         // 0x80808080 when x is uint8 (legalised to int8), else 0
    int32_t ydt;            // 0 uint8, 1 int8 (OUT_REQUANT)
    int32_t lo, hi, zp_y, rounding;
    int32_t y_ldc, y_coff;  // in elements
    int32_t vec_store;      // 1 when 4-element groups of y are 4-element aligned
    int32_t tiles_c;        // channel tiles
    int32_t ntiles;         // tiles_c * pixel tiles
    int32_t nblocks;        // persistent grid size (a multiple of 8)
    int32_t nk;             // K-steps per tile: ceil(J / BK) of the launched kernel
    int32_t mode;           // OutMode of the conv kernel's epilogue
    int32_t fast_rq;        // 1: HALF_UP and every shift in [33, 53] (32-bit requantize)
    int32_t lo_off, hi_off; // output clamp + off (32-bit requantize path)
    uint32_t out_xor;       // 0x80808080 for int8 outputs of the 32-bit path, else 0
    int32_t staged;         // 1: 8-bit output staged through LDS, 16-byte row stores
    int32_t chan_in_lds;    // 1: chan table copied to dynamic LDS (Kpad * 16 bytes)
    uint32_t zp4;           // legalised zp_x in all four bytes (padding value of x')
    // gathers that read zeros for taps outside the image (conv_dma.hip):
    const uint8_t *pcls;    // [M] border class of each output pixel, 255 = interior
    const int32_t *pcorr;   // [classes][Kpad] zp_x * weights of the class's outside taps, or nullptr
    uint32_t mWo, sWo, mHo, sHo;  // magic divisors for m / Wo and t / Ho (mul 0: divisor 1)
    // row-pair mode of conv_dma.hip (S * C4 <= 32): x is the zero-point
    // padded image (H, W padded, pads 0), R counts filter row pairs, S is 1,
    // and row_bytes is the padded image's row stride
    int32_t rowpack, row_bytes;
    // split reduction of the LDS-direct ring kernel: each tile's K-steps in
    // ksplit parts run by separate workgroups; part[] holds their int32
    // partial sums (ntiles * ksplit * TC * TP), cnt[] one arrival counter per
    // tile (zero between launches: the last part resets it)
    int32_t ksplit;
    int32_t *part;
    int32_t *cnt;
    // residual qnn.add fused into the epilogue (staged 8-bit outputs of the
    // kernels that use store_tile): the requantized conv output of channel
    // k at pixel m (dtype ydt) and the residual res[m * r_ldc + r_coff + k]
    // (rdt: 0 uint8, 1 int8) go through add_one(fadd, ., .); the result is
    // stored in place of the conv output.  res == nullptr: no add.
    const uint8_t *res;
    int32_t r_ldc, r_coff, rdt, res_vec;   // res_vec: 16-byte residual rows are 16-byte aligned
    AddArgs fadd;
};

// Depthwise conv arguments (channel multiplier 1).
struct DwArgs {
    const uint8_t *x;
    const int32_t *wq;      // [R*S][C] weights minus zero point, int32 (general kernel)
    const ChanRec *chan;    // [C]: mult, bconst, rndzp, shift (bconst: see the kernels)
    void *y;
    int32_t N, H, W, C, Ho, Wo, R, S;
    int32_t sh, sw, pt, pl, dh, dw;
    int32_t zp_x;           // input zero point in the input's own dtype
    int32_t x_signed;       // 1 when x is int8
    int32_t ydt, lo, hi, zp_y, rounding;
    int32_t y_ldc, y_coff;
    int32_t out_i32;        // 1: raw accumulator output
    // 3x3 dot-product kernel (depthwise.hip)
    const uint32_t *wd;     // [C][3] words (w[r][0][c], w[r][1][c], w[r][2][c], 0)
    const int32_t *zpw;     // [C] weight zero points
    uint32_t flip4;         // 0x80808080 when x is uint8 (legalised to int8), else 0
    uint32_t zp4;           // legalised zp_x in all four bytes (the padding value)
    int32_t zpw_any;        // some weight zero point is not 0 (window sums needed)
    int32_t fast_rq;        // 32-bit requantize (HALF_UP, every shift in [33, 53])
    int32_t lo_off, hi_off; // clamp + off for the 32-bit path
    uint32_t out_xor;       // 0x80808080 for int8 outputs of the 32-bit path
    int32_t vec_store;      // 8-byte output stores allowed
    // LDS-tiled form (band kernel): a workgroup per band of rb output rows
    // and tile of ct strips of one image; the tile's input rows sit in LDS,
    // row stride lrs bytes, LDS column j at byte loff0 + j * C, lcols columns
    int32_t band;           // the band kernel may run (shape and LDS size fit)
    int32_t rb, nband;      // output rows per band, bands per image
    int32_t ct, nct;        // strips per column tile, column tiles per row
    int32_t lrs, loff0, lcols, lbytes, bthreads;
    int32_t seg;            // strips of dw3_pixels() output pixels per work item: 1, 2 or 4
    int32_t items;          // work items: N * Ho * ceil(Wo / (dw3_pixels() * seg)) * C / 8 (< 2^31)
};

// Elementwise requantize / add arguments.
struct ReqArgs {
    const void *x;
    void *y;
    const int32_t *tab;     // per-channel [channels][4] = mult, shift, zp_in, zp_out, or nullptr
    int64_t count;
    int32_t channels;
    int32_t mult, shift, zp_in, zp_out;   // per-tensor values when tab == nullptr
    int32_t lo, hi, rounding;
};


// Tile configurations of the MFMA conv kernel.
enum ConvTile {
    TILE_128x128 = 0,     // 128 channels x 128 pixels, BK 128, 2x2 waves of 64x64
    TILE_64x256 = 1,      // 64 channels x 256 pixels, BK 128, 1x4 waves of 64x64
    TILE_256x128 = 2,     // 256 channels x 128 pixels, BK 128, 2x2 waves of 128x64
    TILE_64x64 = 3,       // 64 x 64, BK 128, 2x2 waves of 32x32
    TILE_64x64_K64 = 4,   // 64 x 64, BK 64 (short reductions, J <= 64)
    TILE_128x128_K64 = 5, // 128 x 128, BK 64
    TILE_128x64 = 6,      // 128 channels x 64 pixels, BK 128, 2x2 waves of 64x32
    TILE_64x128 = 7,      // 64 channels x 128 pixels, BK 128, 2x2 waves of 32x64
    TILE_256x64_K64 = 8,  // 256 channels x 64 pixels, BK 64, 4x1 waves of 64x64
    TILE_COUNT
};

struct TileShape {
    int tc, tp, bk;
};
TileShape tile_shape(int tile);

// Tile configurations of the tap-uniform kernel (conv_tap.hip), used when
// the channel count is a multiple of the K-step: channels x pixels x BK.
enum TapTile {
    TAP_128x128x64 = 0,   // 2x2 waves of 64x64
    TAP_256x128x64 = 1,   // 4x2 waves of 64x64 (512 threads)
    TAP_128x256x64 = 2,   // 2x4 waves of 64x64 (512 threads)
    TAP_128x128x128 = 3,  // 2x2 waves of 64x64
    TAP_256x128x128 = 4,  // 4x2 waves of 64x64 (512 threads)
    TAP_128x256x128 = 5,  // 2x4 waves of 64x64 (512 threads)
    TAP_64x128x128 = 6,   // 1x4 waves of 64x32
    TAP_128x64x128 = 7,   // 4x1 waves of 32x64
    TAP_256x128x128_W4 = 8,  // 2x2 waves of 128x64 (one workgroup per CU)
    TAP_128x256x128_W4 = 9,  // 2x2 waves of 64x128
    TAP_256x128x64_W4 = 10,  // 2x2 waves of 128x64
    TAP_128x256x64_W4 = 11,  // 2x2 waves of 64x128
    TAP_COUNT
};
TileShape tap_tile_shape(int tile);

// Tile configurations of the LDS-direct kernel (conv_dma.hip): channels x
// pixels, wave grid, LDS stages; K-step 64, C % 64 == 0.
enum DmaTile {
    DMA_128x128_S4 = 0,   // 2x2 waves of 64x64, 4 stages
    DMA_128x128_S8 = 1,   // 2x2 waves of 64x64, 8 stages
    DMA_128x64_S4 = 2,    // 2x2 waves of 64x32
    DMA_64x128_S4 = 3,    // 2x2 waves of 32x64
    DMA_64x64_S4 = 4,     // 2x2 waves of 32x32
    DMA_256x128_S4 = 5,   // 4x2 waves of 64x64 (512 threads)
    DMA_128x256_S4 = 6,   // 2x4 waves of 64x64 (512 threads)
    DMA_128x64_S8 = 7,    // 2x2 waves of 64x32, 8 stages
    DMA_256x128_W4 = 8,   // 2x2 waves of 128x64, 4 stages (one workgroup per CU)
    DMA_128x256_W4 = 9,   // 2x2 waves of 64x128, 4 stages
    DMA_128x128_W2A = 10, // 1x2 waves of 128x64, 8 stages
    DMA_128x128_W2B = 11, // 2x1 waves of 64x128, 8 stages
    DMA_64x64_S8 = 12,    // 2x2 waves of 32x32, 8 stages
    DMA_64x128_S8 = 13,   // 2x2 waves of 32x64, 8 stages
    DMA_64x64_S16 = 14,   // 2x2 waves of 32x32, 16 stages (one workgroup per CU)
    // short reductions (J <= 64 * stages): all stages in flight, no ring
    DMA_64x128_R1 = 15,
    DMA_64x64_R1 = 16,
    DMA_128x128_R1 = 17,
    DMA_128x64_R1 = 18,
    DMA_64x128_R2 = 19,
    DMA_128x128_R2 = 20,
    DMA_64x64_R2 = 21,
    DMA_128x64_R2 = 22,
    DMA_64x128_R4 = 23,
    DMA_128x128_R4 = 24,
    DMA_64x64_R4 = 25,
    // two groups of 2x2 waves taking alternate K-steps, 8 stages (4 each)
    DMA_128x64_K2 = 26,
    DMA_64x64_K2 = 27,
    DMA_128x128_K2 = 28,
    DMA_COUNT
};
TileShape dma_tile_shape(int tile);
int dma_threads(int tile);
bool dma_splits(int tile);   // the configuration has a split-reduction form
int dma_split(int tile);    // K-step groups sharing a tile (1 or 2)
int dma_stages(int tile);
int dma_wave_tile(int tile);   // channels x pixels of one wave
bool dma_short(int tile);   // short-reduction form: at most dma_stages(tile) K-steps
hipError_t launch_conv_dma(const ConvArgs &a, int tile, hipStream_t st);
// Wave-independent kernel (conv_wave.hip): 64 x 64 tile per wave, split =
// 1, 2, 4 or 8 waves sharing a tile's reduction (8: 512-thread workgroups).
hipError_t launch_conv_wave(const ConvArgs &a, int split, hipStream_t st);
int wave_threads(int split);
// Window kernel (conv_halo.hip): stride 1, undilated 3x3, C % 64 == 0,
// Wo <= 64; nw = 4 or 8 waves per workgroup, each computing whole output
// rows of one image for 64 channels from an LDS copy of their input window,
// the workgroup's weights resident in LDS.  halo_lds_bytes: dynamic LDS of
// a launch, 0 when the shape is not eligible; halo_pixel_tiles: wave tiles
// per 64-channel tile, -1 when not eligible.
size_t halo_lds_bytes(const ConvArgs &a, int nw);
long long halo_pixel_tiles(const ConvArgs &a);
// 1: the staging tiles have LDS of their own, 0: they reuse the window's
// (-1: not eligible)
int halo_layout(const ConvArgs &a, int nw);
hipError_t launch_conv_halo(const ConvArgs &a, int nw, hipStream_t st);
// Streaming window kernel (conv_window.hip): stride 1, undilated 3x3,
// C % 64 == 0, Wo <= 64; the input window of a workgroup's bands stays in
// LDS while the weights stream through it.  cfg indexes its configurations
// (bands per workgroup, reduction split, channels per workgroup).
int win_count();
int win_channels(int cfg);
int win_threads(int cfg);
size_t win_lds_bytes(const ConvArgs &a, int cfg);               // 0: not eligible
long long win_workgroups_per_ctile(const ConvArgs &a, int cfg);  // -1: not eligible
hipError_t launch_conv_window(const ConvArgs &a, int cfg, hipStream_t st);
hipError_t launch_frag_pack(const int8_t *wp, int Kpad, int Jpad, int8_t *out, hipStream_t st);
// corr[c][k] = zp_x * (sum of packed weights of row k over the taps outside
// the image in border class c: tap (r, s) is inside when bit r of rmask[c]
// and bit s of cmask[c] are set).
hipError_t launch_rowpack_weights(const int8_t *w, int K, int R, int S, int C, int C4, int Kpad, int Jpad, int8_t *wp,
                                  hipStream_t st);
hipError_t launch_pad_image(const uint8_t *x, int N, int H, int W, int C, int Hp, int Wp, int C4, int pt, int pl,
                            uint8_t zp, uint8_t *out, hipStream_t st);
hipError_t launch_border_corr(const int8_t *wp, int Kpad, int Jpad, int C4, int S, int RS, const uint32_t *rmask,
                              const uint32_t *cmask, int ncls, int32_t zpx, int32_t *corr, hipStream_t st);
int tap_threads(int tile);
int tap_wave_tile(int tile);   // channels x pixels of one wave
hipError_t launch_conv_tap(const ConvArgs &a, int tile, hipStream_t st);

// Activation gather width in bytes: 16 when C % 16 == 0, 8 when C % 8 == 0,
// else 4 (C % 4 == 0 after channel padding).
int gather_width(int C);

hipError_t launch_conv(const ConvArgs &a, int tile, int avec, hipStream_t st);
// Resident workgroups per CU of a conv kernel instantiation (occupancy),
// given its dynamic LDS bytes.
int conv_blocks_per_cu(int tile, int avec, size_t dyn_lds);
hipError_t launch_window_sums(const ConvArgs &a, int32_t *out, hipStream_t st);
hipError_t launch_pad_channels(const uint8_t *x, uint8_t *xp, long long pixels, int C, int C4, uint8_t zp,
                               hipStream_t st);
hipError_t launch_prep_conv(const int8_t *w, const int32_t *bias, int K, int RS, int C, int C4, int Jpad,
                            int Kpad, int32_t zpx, int8_t *wp, ChanRec *chan, const int32_t *zpw, hipStream_t st);
hipError_t launch_prep_dw(const int8_t *w, const int32_t *bias, int RS, int C, const int32_t *zpw, int32_t *wq,
                          ChanRec *chan, hipStream_t st);
hipError_t launch_depthwise(const DwArgs &a, hipStream_t st);
// 3x3, undilated, C % 8 == 0, stride_w 1 or 2, x 8-byte aligned
hipError_t launch_prep_dw3(const int8_t *w, const int32_t *bias, int C, int32_t zpx_l, const int32_t *zpw,
                           uint32_t *wd, ChanRec *chan, hipStream_t st);
hipError_t launch_depthwise3(const DwArgs &a, hipStream_t st);
int dw3_pixels();   // output pixels along a row per work item of launch_depthwise3
hipError_t launch_depthwise3_band(const DwArgs &a, hipStream_t st);
hipError_t launch_requantize(const ReqArgs &a, int xdt, int ydt, bool aligned, hipStream_t st);
// Reads `bytes` (a multiple of 16) of `buf` through the caches (kernel
// tuning uses it to evict what a timed launch would otherwise find cached).
hipError_t launch_cache_sweep(const void *buf, size_t bytes, int *sink, hipStream_t st);
hipError_t launch_flip_bytes(const uint8_t *in, uint8_t *out, size_t n, hipStream_t st);
hipError_t launch_add(const AddArgs &a, int adt, int bdt, int ydt, bool aligned, hipStream_t st);
// Builds AddArgs::tab (512 int32) for operand dtypes adt and bdt (0 uint8, 1 int8).
hipError_t launch_add_table(const AddArgs &a, int adt, int bdt, int32_t *tab, hipStream_t st);

// Quantized pool2d (Eq. (4)): NHWC input and output of one dtype; mode 0
// average (rounding 0 HALF_UP, 1 HALF_AWAY; count_pad counts padded cells
// as zp), mode 1 max.  vec is 16, 4 or 1 channels per thread (C a multiple
// of vec, x and y aligned to vec bytes).
struct PoolArgs {
    const void *x;
    void *y;
    int N, H, W, C, R, S, sh, sw, pt, pl, Ho, Wo;
    int mode, count_pad, zp, rounding;
};
hipError_t launch_pool(const PoolArgs &a, bool is_signed, int vec, hipStream_t st);
// The window-split form for few output pixels with large windows: one
// workgroup per output pixel and 64*vec channels (vec 4 or 1).
hipError_t launch_pool_split(const PoolArgs &a, bool is_signed, int vec, hipStream_t st);

}  // namespace qnn
