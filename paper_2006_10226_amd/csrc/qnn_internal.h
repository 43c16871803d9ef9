// Internal declarations shared by the host side of libqnn (qnn_api.cpp) and
// its HIP kernels.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qnn {

// Per-output-channel epilogue record of a conv / dense plan.
//   mult, shift : fixed-point requantize multiplier (shift clamped to <= 63;
//                 every product with shift >= 63 rounds to 0 anyway)
//   bconst      : bias[k] - zp_x' * sum_j w[k,j] + J * zp_x' * zp_w[k]
//                 (terms 2 and 4 of Eq. (3) folded with the bias; int32
//                 wrap-around arithmetic, exact whenever the true result
//                 fits int32, which plan creation guarantees)
//   zpw         : weight zero point (term 3 coefficient)
struct ChanRec {
    int32_t mult, shift, bconst, zpw;
};

enum OutMode { OUT_REQUANT = 0, OUT_INT32 = 1, OUT_PARTIAL = 2 };

// Implicit-GEMM conv arguments.  GEMM view: D[k][m] = sum_j Wp[k][j] * X'[m][j]
// with m = output pixel, k = output channel, j = (r*S + s)*C + c.
struct ConvArgs {
    const uint8_t *x;       // NHWC activations (uint8 or int8 bytes)
    const int8_t *wp;       // packed weights [Kpad][Jpad], zero padded
    const ChanRec *chan;    // [Kpad]
    const int32_t *asum;    // [M] window sums of x' (term 3) or nullptr
    void *y;                // output (requantized bytes or int32)
    int32_t *ws;            // split-K partials [nsplit][M][Kpad]
    int32_t N, H, W, C, Ho, Wo, R, S;
    int32_t sh, sw, pt, pl, dh, dw;
    int32_t K, Kpad, J, Jpad, M;
    uint32_t flip4;         // 0x80808080 when x is uint8 (legalised to int8), else 0
    uint32_t pad4;          // padding byte zp_x' replicated 4 times
    int32_t ydt;            // 0 uint8, 1 int8 (OUT_REQUANT)
    int32_t lo, hi, zp_y, rounding;
    int32_t y_ldc, y_coff;  // in elements
    int32_t vec_store;      // 1 when 4-element groups of y are 4-element aligned
    int32_t ksteps;         // K-steps (of the tile's BK) per split
    int32_t nsplit;
    int32_t tiles_c;        // channel tiles
    int32_t nblocks;        // tiles_c * pixel tiles
};

// Depthwise conv arguments (channel multiplier 1).
struct DwArgs {
    const uint8_t *x;
    const int32_t *wq;      // [R*S][C] weights minus zero point, int32
    const ChanRec *chan;    // [C]: mult, shift, bconst (= bias), unused
    void *y;
    int32_t N, H, W, C, Ho, Wo, R, S;
    int32_t sh, sw, pt, pl, dh, dw;
    int32_t zp_x;           // input zero point in the input's own dtype
    int32_t x_signed;       // 1 when x is int8
    int32_t ydt, lo, hi, zp_y, rounding;
    int32_t y_ldc, y_coff;
    int32_t out_i32;        // 1: raw accumulator output
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

struct AddArgs {
    const void *a;
    const void *b;
    void *y;
    int64_t count;
    int32_t ma, na, zpa, mb, nb, zpb, zp_y;
    int32_t lo, hi, rounding;
};

// Tile configurations of the MFMA conv kernel.
enum ConvTile {
    TILE_128x128 = 0,   // 128 channels x 128 pixels, 2x2 waves of 64x64
    TILE_64x256 = 1,    // 64 channels x 256 pixels, 1x4 waves of 64x64
    TILE_256x128 = 2,   // 256 channels x 128 pixels, 2x2 waves of 128x64
    TILE_64x64 = 3,     // 64 x 64, 2x2 waves of 32x32 (small problems)
    TILE_COUNT
};

struct TileShape {
    int tc, tp, bk;
};
TileShape tile_shape(int tile);

// Activation gather width in bytes: 16 when C % 16 == 0, else 4 when
// C % 4 == 0, else 1.
int gather_width(int C);

hipError_t launch_conv(const ConvArgs &a, int tile, int avec, int mode, hipStream_t st);
hipError_t launch_splitk_reduce(const ConvArgs &a, int mode, hipStream_t st);
hipError_t launch_window_sums(const ConvArgs &a, int32_t *out, hipStream_t st);
hipError_t launch_prep_conv(const int8_t *w, const int32_t *bias, int K, int J, int Jpad,
                            int Kpad, int32_t zpx, int8_t *wp, ChanRec *chan, hipStream_t st);
hipError_t launch_prep_dw(const int8_t *w, const int32_t *bias, int RS, int C, int32_t *wq,
                          ChanRec *chan, hipStream_t st);
hipError_t launch_depthwise(const DwArgs &a, hipStream_t st);
hipError_t launch_requantize(const ReqArgs &a, int xdt, int ydt, bool aligned, hipStream_t st);
hipError_t launch_add(const AddArgs &a, int adt, int bdt, int ydt, bool aligned, hipStream_t st);

}  // namespace qnn
