// 3x3 depthwise quantized conv (channel multiplier 1) on 4-way int8 dot
// products, with the requantize of Eq. (5) fused.
//
// Arithmetic: the four-term expansion of Eq. (3) per channel (Jain et al.,
// Sec. II-B, III-B) with the sum running over the 9 taps of one channel:
//   sum_t (x~'_t - zp')(w_t - zp_w) = sum_t x~'_t w_t - zp_w sum_t x~'_t
//                                     - zp' sum_t w_t + 9 zp' zp_w
// x' is the activation legalised to int8 (uint8 XOR 0x80, Sec. III-C), x~'
// is x' inside the image and zp' on padded taps.  The last two terms and
// the bias are one per-channel constant (ChanRec.bconst of the plan); the
// first is a v_dot4_i32_i8 per filter row over a word holding the three
// taps of that row for one channel (the weight word carries 0 in its
// fourth byte); the second is only computed when a weight zero point is
// not 0.
//
// Work item: 8 channels (one 8-byte load per input pixel) x P output
// pixels along a row.  The weights of the 8 channels stay in registers as
// 24 words; the input columns of the strip are loaded once per filter row
// and turned into per-channel tap words with byte permutes (for stride 1
// the word of pixel p + 1 is one permute of the word of pixel p).  The
// kernel reads every input byte a few times from L2 and once from HBM,
// writes every output byte once, and is bound by HBM.
#include "qnn_internal.h"

namespace qnn {

namespace {

__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel)
{
    return __builtin_amdgcn_perm(hi, lo, sel);
}

__device__ __forceinline__ int dot4(uint32_t a, uint32_t b, int c)
{
    return __builtin_amdgcn_sdot4((int)a, (int)b, c, false);
}

// cache policy of the output stores: nt, the streaming hint (the output is
// written once; it need not stay in this XCD's L2)
constexpr int kStream = 2;

// byte selector of v_perm_b32: 0..3 bytes of `lo`, 4..7 bytes of `hi`,
// 12 a zero byte
constexpr uint32_t kZero = 0x0c;

}  // namespace

// output pixels per work item
constexpr int kDw3Pixels = 4;

// OUT: 0 = requantized bytes, 32-bit rounding shift (HALF_UP, every shift
// in [33, 53]); 1 = requantized bytes, 64-bit rounding shift; 2 = int32.
template <int SW, int P, bool ZPW, int OUT>
__global__ void __launch_bounds__(256) depthwise3_kernel(DwArgs a)
{
    constexpr int NCOL = (P - 1) * SW + 3;      // input columns of the strip
    // work item index < 2^31 and every byte offset < 2^31 (host checks):
    // 32-bit index arithmetic and buffer addressing throughout
    const unsigned nch = (unsigned)a.C >> 3;
    const unsigned nstrip = ((unsigned)a.Wo + P - 1) / P;
    // workgroups are dealt to the 8 XCDs round-robin and each XCD has its
    // own L2: XCD x takes the x-th eighth of the work list (the grid is a
    // multiple of 8), so the output rows that share input rows run on one
    // XCD and the input is fetched from HBM about once
    const unsigned lb = (blockIdx.x & 7u) * (gridDim.x >> 3) + (blockIdx.x >> 3);
    const unsigned gid = lb * blockDim.x + threadIdx.x;
    if (gid >= (unsigned)a.items)
        return;
    const unsigned chunk = gid % nch;
    unsigned rest = gid / nch;
    const unsigned strip = rest % nstrip;
    rest /= nstrip;
    const int oh = (int)(rest % (unsigned)a.Ho);
    const int n = (int)(rest / (unsigned)a.Ho);
    const int c0 = (int)chunk * 8;
    const int ow0 = (int)strip * P;

    const __amdgpu_buffer_rsrc_t rx =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.x, (short)0, a.N * a.H * a.W * a.C, 0x00020000);

    // weight words of the 8 channels: wd[c][r] = (w[r][0][c], w[r][1][c], w[r][2][c], 0)
    uint32_t wv[8][3];
#pragma unroll
    for (int i = 0; i < 6; ++i) {
        const uint4 q = ((const uint4 *)(a.wd + (size_t)c0 * 3))[i];
        const uint32_t d[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int e = 0; e < 4; ++e)
            wv[(4 * i + e) / 3][(4 * i + e) % 3] = d[e];
    }

    int acc[8][P], xs[8][P];
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
        for (int p = 0; p < P; ++p) {
            acc[c][p] = 0;
            xs[c][p] = 0;
        }

#pragma unroll
    for (int r = 0; r < 3; ++r) {
        const int ih = oh * a.sh - a.pt + r;
        const bool row_in = (unsigned)ih < (unsigned)a.H;
        const int rowoff = (n * a.H + min(max(ih, 0), a.H - 1)) * a.W * a.C + c0;
        // every column is loaded (clamped into the image) and replaced by
        // the padding value where it lies outside
        uint32_t D[NCOL][2];
#pragma unroll
        for (int q = 0; q < NCOL; ++q) {
            const int iw = ow0 * SW - a.pl + q;
            const bool in = row_in && (unsigned)iw < (unsigned)a.W;
            const int off = rowoff + min(max(iw, 0), a.W - 1) * a.C;
            const auto v = __builtin_amdgcn_raw_buffer_load_b64(rx, off, 0, 0);
            D[q][0] = in ? (uint32_t)v[0] ^ a.flip4 : a.zp4;
            D[q][1] = in ? (uint32_t)v[1] ^ a.flip4 : a.zp4;
        }
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const int h = c >> 2;
            const uint32_t b = (uint32_t)(c & 3);
            uint32_t cw = 0;
#pragma unroll
            for (int p = 0; p < P; ++p) {
                if (SW == 1 && p > 0) {
                    // slide: bytes 1, 2 of the previous word, then the new column
                    cw = perm(D[p + 2][h], cw, 1u | (2u << 8) | ((4u + b) << 16) | (kZero << 24));
                } else {
                    const int q = p * SW;
                    const uint32_t t = perm(D[q + 1][h], D[q][h], b | ((4u + b) << 8) | (kZero << 16) | (kZero << 24));
                    cw = perm(D[q + 2][h], t, 0u | (1u << 8) | ((4u + b) << 16) | (kZero << 24));
                }
                acc[c][p] = dot4(cw, wv[c][r], acc[c][p]);
                if constexpr (ZPW)
                    xs[c][p] = dot4(cw, 0x00010101u, xs[c][p]);
            }
        }
    }

    // epilogue: constant terms, requantize, store
    ChanRec cr[8];
#pragma unroll
    for (int c = 0; c < 8; ++c)
        cr[c] = a.chan[c0 + c];
    int zw[8];
#pragma unroll
    for (int c = 0; c < 8; ++c)
        zw[c] = ZPW ? a.zpw[c0 + c] : 0;
    const __amdgpu_buffer_rsrc_t ry = __builtin_amdgcn_make_buffer_rsrc(a.y, (short)0, 0x7fffffff, 0x00020000);
#pragma unroll
    for (int p = 0; p < P; ++p) {
        const int ow = ow0 + p;
        if (ow >= a.Wo)
            break;
        const int m = (n * a.Ho + oh) * a.Wo + ow;
        int v[8];
#pragma unroll
        for (int c = 0; c < 8; ++c)
            v[c] = (int)((uint32_t)acc[c][p] + (uint32_t)cr[c].bconst - (uint32_t)(zw[c] * xs[c][p]));
        if constexpr (OUT == 2) {
            const int off = (m * a.y_ldc + a.y_coff + c0) * 4;
#pragma unroll
            for (int c = 0; c < 8; ++c)
                __builtin_amdgcn_raw_buffer_store_b32(v[c], ry, off + 4 * c, 0, kStream);
            continue;
        }
        uint32_t packed[2] = {0u, 0u};
        if constexpr (OUT == 0) {
            // 32-bit form of the rounding shift: rndzp carries
            // 2^(sh-1) + (zp_y + off) 2^sh with sh = shift - 32
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                const int t = (__mulhi(v[c], cr[c].mult) + cr[c].rndzp) >> (cr[c].shift & 31);   // shift - 32
                packed[c >> 2] |= (uint32_t)clamp_i32(t, a.lo_off, a.hi_off) << (8 * (c & 3));
            }
            packed[0] ^= a.out_xor;
            packed[1] ^= a.out_xor;
        } else {
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                long long o = rounding_mul_shift(v[c], cr[c].mult, cr[c].shift, a.rounding) + a.zp_y;
                o = o < a.lo ? a.lo : (o > a.hi ? a.hi : o);
                packed[c >> 2] |= ((uint32_t)o & 0xffu) << (8 * (c & 3));
            }
        }
        const int off = m * a.y_ldc + a.y_coff + c0;
        if (a.vec_store) {
            __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(__attribute__((ext_vector_type(2))) unsigned,
                                                                     uint2{packed[0], packed[1]}),
                                                  ry, off, 0, kStream);
        } else {
#pragma unroll
            for (int c = 0; c < 8; ++c)
                __builtin_amdgcn_raw_buffer_store_b8((uint8_t)(packed[c >> 2] >> (8 * (c & 3))), ry, off + c, 0,
                                                     kStream);
        }
    }
}

// Plan preparation, one thread per channel: the three weight words and the
// constant bias - zp' sum_t w_t + 9 zp' zp_w[c] (Eq. (3) terms 2 and 4 plus
// the bias, in wrapping int32 like the accumulator).  w is [3][3][C].
__global__ void __launch_bounds__(256) prep_dw3_kernel(const int8_t *w, const int32_t *bias, int C, int32_t zpx_l,
                                                       const int32_t *zpw, uint32_t *wd, ChanRec *chan)
{
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= C)
        return;
    int wsum = 0;
    for (int r = 0; r < 3; ++r) {
        uint32_t word = 0;
        for (int s = 0; s < 3; ++s) {
            const int8_t v = w[(r * 3 + s) * C + c];
            wsum += v;
            word |= (uint32_t)(uint8_t)v << (8 * s);
        }
        wd[(size_t)c * 3 + r] = word;
    }
    const uint32_t b = bias ? (uint32_t)bias[c] : 0u;
    chan[c].bconst = (int)(b - (uint32_t)zpx_l * (uint32_t)wsum + 9u * (uint32_t)zpx_l * (uint32_t)zpw[c]);
}

hipError_t launch_prep_dw3(const int8_t *w, const int32_t *bias, int C, int32_t zpx_l, const int32_t *zpw,
                           uint32_t *wd, ChanRec *chan, hipStream_t st)
{
    hipLaunchKernelGGL(prep_dw3_kernel, dim3((C + 255) / 256), dim3(256), 0, st, w, bias, C, zpx_l, zpw, wd, chan);
    return hipGetLastError();
}

template <int SW, bool ZPW, int OUT>
static void launch_dw3_cfg(const DwArgs &a, dim3 grid, hipStream_t st)
{
    launch_main((depthwise3_kernel<SW, kDw3Pixels, ZPW, OUT>), grid, dim3(256), 0, st, a);
}

template <int SW, bool ZPW>
static void launch_dw3_out(const DwArgs &a, dim3 grid, hipStream_t st)
{
    if (a.out_i32)
        launch_dw3_cfg<SW, ZPW, 2>(a, grid, st);
    else if (a.fast_rq)
        launch_dw3_cfg<SW, ZPW, 0>(a, grid, st);
    else
        launch_dw3_cfg<SW, ZPW, 1>(a, grid, st);
}

hipError_t launch_depthwise3(const DwArgs &a, hipStream_t st)
{
    if (a.R != 3 || a.S != 3 || a.dh != 1 || a.dw != 1 || a.C % 8 != 0 || a.sh < 1 || (a.sw != 1 && a.sw != 2))
        return hipErrorInvalidValue;
    if (a.items == 0)
        return hipSuccess;
    const dim3 grid((unsigned)(((a.items + 255) / 256 + 7) / 8 * 8));
    if (a.sw == 1)
        a.zpw_any ? launch_dw3_out<1, true>(a, grid, st) : launch_dw3_out<1, false>(a, grid, st);
    else
        a.zpw_any ? launch_dw3_out<2, true>(a, grid, st) : launch_dw3_out<2, false>(a, grid, st);
    return hipGetLastError();
}

int dw3_pixels()
{
    return kDw3Pixels;
}

}  // namespace qnn
