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
// Work item: 8 channels (one 8-byte load per input pixel) x a segment of
// T strips of P output pixels along a row.  The weights and per-channel
// records of the 8 channels stay in registers for the whole segment; the
// input columns are loaded once per filter row as the segment slides along
// (a strip reuses the last columns of the one before it) and turned into
// per-channel tap words with byte permutes (for stride 1 the word of pixel
// p + 1 is one permute of the word of pixel p, carried across strips).
// The kernel reads every input byte about once from L2 and once from HBM,
// writes every output byte once, and is bound by HBM and by its VALU
// work (about three dot products, three permutes and the requantize per
// output).
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

// output pixels per strip
constexpr int kDw3Pixels = 4;

// OUT: 0 = requantized bytes, 32-bit rounding shift (HALF_UP, every shift
// in [33, 53]); 1 = requantized bytes, 64-bit rounding shift; 2 = int32.
template <int SW, int P, int T, bool ZPW, int OUT>
__global__ void __launch_bounds__(256) depthwise3_kernel(DwArgs a)
{
    constexpr int NCOL = (P - 1) * SW + 3;   // input columns of one strip
    constexpr int STEP = P * SW;             // columns between the starts of two strips
    constexpr int KEEP = NCOL - STEP;        // columns a strip shares with the next
    // work item index < 2^31 and every in-image byte offset < 2^31 (host
    // checks): 32-bit index arithmetic and buffer addressing throughout;
    // offsets of taps outside the image may wrap, and those loads are
    // replaced by the padding value (a wrapped offset lies past the end of
    // the buffer, where buffer loads return zeros)
    const unsigned nch = (unsigned)a.C >> 3;
    const unsigned nseg = ((unsigned)a.Wo + P * T - 1) / (P * T);
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
    const unsigned seg = rest % nseg;
    rest /= nseg;
    const int oh = (int)(rest % (unsigned)a.Ho);
    const int n = (int)(rest / (unsigned)a.Ho);
    const int c0 = (int)chunk * 8;
    const int ow0 = (int)seg * (P * T);

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
    ChanRec cr[8];
#pragma unroll
    for (int c = 0; c < 8; ++c)
        cr[c] = a.chan[c0 + c];
    int zw[8];
#pragma unroll
    for (int c = 0; c < 8; ++c)
        zw[c] = ZPW ? a.zpw[c0 + c] : 0;

    // rows of the filter: base offset of column 0 of the segment, and
    // whether the row lies inside the image
    const int cw0 = ow0 * SW - a.pl;   // input column of the segment's first tap
    unsigned rowoff[3];
    bool row_in[3];
#pragma unroll
    for (int r = 0; r < 3; ++r) {
        const int ih = oh * a.sh - a.pt + r;
        row_in[r] = (unsigned)ih < (unsigned)a.H;
        rowoff[r] = ((unsigned)(n * a.H + ih) * (unsigned)a.W + (unsigned)cw0) * (unsigned)a.C + (unsigned)c0;
    }
    // column q of the segment, row r: two words of 4 legalised channels
    auto load_col = [&](int r, int q, uint32_t (&d)[2]) {
        const bool in = row_in[r] && (unsigned)(cw0 + q) < (unsigned)a.W;
        const auto v = __builtin_amdgcn_raw_buffer_load_b64(rx, (int)(rowoff[r] + (unsigned)q * (unsigned)a.C), 0, 0);
        d[0] = in ? (uint32_t)v[0] ^ a.flip4 : a.zp4;
        d[1] = in ? (uint32_t)v[1] ^ a.flip4 : a.zp4;
    };

    const __amdgpu_buffer_rsrc_t ry = __builtin_amdgcn_make_buffer_rsrc(a.y, (short)0, 0x7fffffff, 0x00020000);
    const int m0 = (n * a.Ho + oh) * a.Wo + ow0;

    // carried from strip to strip: the last KEEP columns of each row and,
    // for stride 1, the tap word of each row's last pixel
    uint32_t D[3][NCOL][2];
    uint32_t cwc[3][8];
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
        for (int c = 0; c < 8; ++c)
            cwc[r][c] = 0;

#pragma unroll
    for (int t = 0; t < T; ++t) {
        if (ow0 + t * P >= a.Wo)
            break;
        // the strip's new input columns (the first strip loads them all)
#pragma unroll
        for (int r = 0; r < 3; ++r) {
            if (t > 0) {
#pragma unroll
                for (int k = 0; k < KEEP; ++k) {
                    D[r][k][0] = D[r][k + STEP][0];
                    D[r][k][1] = D[r][k + STEP][1];
                }
            }
#pragma unroll
            for (int q = (t > 0 ? KEEP : 0); q < NCOL; ++q)
                load_col(r, t * STEP + q, D[r][q]);
        }

        int acc[8][P], xs[8][P];
#pragma unroll
        for (int r = 0; r < 3; ++r) {
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                const int h = c >> 2;
                const uint32_t b = (uint32_t)(c & 3);
                uint32_t cw = cwc[r][c];
#pragma unroll
                for (int p = 0; p < P; ++p) {
                    if (SW == 1 && (p > 0 || t > 0)) {
                        // slide: bytes 1, 2 of the previous word, then the new column
                        cw = perm(D[r][p + 2][h], cw, 1u | (2u << 8) | ((4u + b) << 16) | (kZero << 24));
                    } else {
                        const int q = p * SW;
                        const uint32_t u =
                            perm(D[r][q + 1][h], D[r][q][h], b | ((4u + b) << 8) | (kZero << 16) | (kZero << 24));
                        cw = perm(D[r][q + 2][h], u, 0u | (1u << 8) | ((4u + b) << 16) | (kZero << 24));
                    }
                    // the first filter row starts from the per-channel constant
                    acc[c][p] = dot4(cw, wv[c][r], r == 0 ? cr[c].bconst : acc[c][p]);
                    if constexpr (ZPW)
                        xs[c][p] = dot4(cw, 0x00010101u, r == 0 ? 0 : xs[c][p]);
                }
                cwc[r][c] = cw;
            }
        }

        // epilogue: requantize and store the strip
#pragma unroll
        for (int p = 0; p < P; ++p) {
            const int ow = ow0 + t * P + p;
            if (ow >= a.Wo)
                break;
            const int m = m0 + t * P + p;
            int v[8];
#pragma unroll
            for (int c = 0; c < 8; ++c)
                v[c] = ZPW ? (int)((uint32_t)acc[c][p] - (uint32_t)(zw[c] * xs[c][p])) : acc[c][p];
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
                    const int u = (__mulhi(v[c], cr[c].mult) + cr[c].rndzp) >> (cr[c].shift & 31);   // shift - 32
                    packed[c >> 2] |= (uint32_t)clamp_i32(u, a.lo_off, a.hi_off) << (8 * (c & 3));
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
                __builtin_amdgcn_raw_buffer_store_b64(
                    __builtin_bit_cast(__attribute__((ext_vector_type(2))) unsigned, uint2{packed[0], packed[1]}), ry,
                    off, 0, kStream);
            } else {
#pragma unroll
                for (int c = 0; c < 8; ++c)
                    __builtin_amdgcn_raw_buffer_store_b8((uint8_t)(packed[c >> 2] >> (8 * (c & 3))), ry, off + c, 0,
                                                         kStream);
            }
        }
    }
}

// LDS-tiled form.  A workgroup takes a band of rb output rows of one image
// and a tile of ct strips of P output columns: the input rows and columns
// the tile reads are copied into LDS with 16-byte LDS-direct loads (each
// wave instruction moves 1 KB of one row, so the reads are whole cache
// lines and need no registers), the padding cells are filled with zp_x,
// and each thread then walks one strip of P output pixels x 4 channels
// down the whole band.  Moving down one output row (stride 1) brings one
// new input row: the tap words of the other two are kept from the rows
// above, so every input row is read from LDS and turned into tap words
// once.  Requires C % 8 == 0, W * C % 16 == 0, x 16-byte aligned and, with
// more than one column tile, C % 16 == 0 (the host checks); vertical
// stride 1 or 2.
template <int SW, int SH, bool FLIP, bool ZPW, int OUT>
__global__ void __launch_bounds__(512) depthwise3_band_kernel(DwArgs a)
{
    extern __shared__ __attribute__((aligned(16))) int8_t tile[];
    constexpr int P = kDw3Pixels;
    constexpr int NCOL = (P - 1) * SW + 3;   // input columns of one strip
    const unsigned nwg = (unsigned)a.N * (unsigned)a.nband * (unsigned)a.nct;
    // XCD x takes the x-th eighth of the tiles (grid a multiple of 8)
    const unsigned wg = (blockIdx.x & 7u) * (gridDim.x >> 3) + (blockIdx.x >> 3);
    if (wg >= nwg)
        return;   // the whole workgroup
    const int C = a.C;
    const int ctile = (int)(wg % (unsigned)a.nct);
    const unsigned nb = wg / (unsigned)a.nct;
    const int n = (int)(nb / (unsigned)a.nband);
    const int oh0 = (int)(nb % (unsigned)a.nband) * a.rb;
    const int rows = min(a.rb, a.Ho - oh0);
    const int nr = (rows - 1) * SH + 3;       // input rows of the band
    const int ih0 = oh0 * SH - a.pt;
    const int ow_t = ctile * a.ct * P;        // first output column of the tile
    const int j0 = ow_t * SW - a.pl;          // image column of LDS column 0
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nwave = (int)(blockDim.x >> 6);

    // 1. the tile's image columns of each input row, 1 KB per wave
    // instruction; lane L writes bytes 16 L .. 16 L + 15 of the block (lanes
    // past the run's end issue nothing)
    const int ic0 = max(j0, 0), ic1 = min(j0 + a.lcols, a.W);
    const int runbytes = max(ic1 - ic0, 0) * C;   // a multiple of 16
    const int nblk = (runbytes + 1023) >> 10;
    const int dst0 = a.loff0 + (ic0 - j0) * C;    // 16-aligned
    const __amdgpu_buffer_rsrc_t rx =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.x, (short)0, a.N * a.H * a.W * C, 0x00020000);
    for (int task = wave; task < nr * nblk; task += nwave) {
        const int r = task / nblk, k = task - r * nblk;
        const int ih = ih0 + r;
        if ((unsigned)ih >= (unsigned)a.H)
            continue;   // padding row: filled below
        const int byte = k * 1024 + lane * 16;
        if (byte < runbytes)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rx, (__attribute__((address_space(3))) void *)(tile + r * a.lrs + dst0 + k * 1024), 16,
                ((n * a.H + ih) * a.W + ic0) * C + byte, 0, 0, 0);
    }

    // 2. the padding cells: columns outside the image in image rows, every
    // column of the rows outside it (raw bytes: the reads below legalise)
    const uint32_t zraw = FLIP ? a.zp4 ^ a.flip4 : a.zp4;
    const uint2 z2 = {zraw, zraw};
    const int cu = C >> 3;                     // 8-byte units per column
    const int lpad = min(max(-j0, 0), a.lcols);            // LDS columns left of the image
    const int rfirst = max(min(a.W - j0, a.lcols), lpad);  // first LDS column right of it
    const int npc = lpad + (a.lcols - rfirst);
    for (int u = tid; u < nr * npc * cu; u += blockDim.x) {
        const int r = u / (npc * cu), rest = u - r * (npc * cu);
        const int jj = rest / cu, e = rest - jj * cu;
        const int j = jj < lpad ? jj : rfirst + (jj - lpad);
        *(uint2 *)(tile + r * a.lrs + a.loff0 + j * C + 8 * e) = z2;
    }
    for (int r = 0; r < nr; ++r) {
        if ((unsigned)(ih0 + r) < (unsigned)a.H)
            continue;
        for (int u = tid; u < a.lcols * cu; u += blockDim.x)
            *(uint2 *)(tile + r * a.lrs + a.loff0 + 8 * u) = z2;
    }
    // vmcnt(0): this wave's LDS-direct loads have landed
    __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (15 << 8));
    __syncthreads();

    // 3. strips of P pixels x 4 channels, each down the whole band
    const int nq = C >> 2;
    const int nstrip = min(a.ct, (a.Wo - ow_t + P - 1) / P);   // strips of this tile
    const __amdgpu_buffer_rsrc_t ry = __builtin_amdgcn_make_buffer_rsrc(a.y, (short)0, 0x7fffffff, 0x00020000);
    for (int it = tid; it < nq * nstrip; it += blockDim.x) {
        const int q = it % nq, strip = it / nq;
        const int c0 = q * 4, ow0 = ow_t + strip * P;
        // weight words of the 4 channels (w[r][0][c], w[r][1][c], w[r][2][c], 0)
        uint32_t wv[4][3];
        {
            const uint4 *wp = (const uint4 *)(a.wd + (size_t)c0 * 3);
            const uint4 w0 = wp[0], w1 = wp[1], w2 = wp[2];
            const uint32_t d[12] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w, w2.x, w2.y, w2.z, w2.w};
#pragma unroll
            for (int i = 0; i < 12; ++i)
                wv[i / 3][i % 3] = d[i];
        }
        ChanRec cr[4];
#pragma unroll
        for (int c = 0; c < 4; ++c)
            cr[c] = a.chan[c0 + c];
        int zw[4];
#pragma unroll
        for (int c = 0; c < 4; ++c)
            zw[c] = ZPW ? a.zpw[c0 + c] : 0;
        const int8_t *col0 = tile + a.loff0 + strip * P * SW * C + c0;

        // tap words of LDS row lr: T[c][p] = (x[p*SW], x[p*SW+1], x[p*SW+2], 0) of channel c
        auto taps = [&](int lr, uint32_t (&T)[4][P]) {
            uint32_t d[NCOL];
            const int8_t *rp = col0 + lr * a.lrs;
#pragma unroll
            for (int k = 0; k < NCOL; ++k)
                d[k] = *(const uint32_t *)(rp + k * C) ^ (FLIP ? a.flip4 : 0u);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const uint32_t b = (uint32_t)c;
#pragma unroll
                for (int p = 0; p < P; ++p) {
                    if (SW == 1 && p > 0) {
                        T[c][p] = perm(d[p + 2], T[c][p - 1], 1u | (2u << 8) | ((4u + b) << 16) | (kZero << 24));
                    } else {
                        const int k = p * SW;
                        const uint32_t u = perm(d[k + 1], d[k], b | ((4u + b) << 8) | (kZero << 16) | (kZero << 24));
                        T[c][p] = perm(d[k + 2], u, 0u | (1u << 8) | ((4u + b) << 16) | (kZero << 24));
                    }
                }
            }
        };
        // output row o of the band from the tap words of its three input rows
        auto out_row = [&](int o, const uint32_t (&T0)[4][P], const uint32_t (&T1)[4][P], const uint32_t (&T2)[4][P]) {
            const int m0 = (n * a.Ho + oh0 + o) * a.Wo + ow0;
#pragma unroll
            for (int p = 0; p < P; ++p) {
                if (ow0 + p >= a.Wo)
                    break;
                int v[4];
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    int acc = dot4(T0[c][p], wv[c][0], cr[c].bconst);
                    acc = dot4(T1[c][p], wv[c][1], acc);
                    acc = dot4(T2[c][p], wv[c][2], acc);
                    if constexpr (ZPW) {
                        int xs = dot4(T0[c][p], 0x00010101u, 0);
                        xs = dot4(T1[c][p], 0x00010101u, xs);
                        xs = dot4(T2[c][p], 0x00010101u, xs);
                        acc = (int)((uint32_t)acc - (uint32_t)(zw[c] * xs));
                    }
                    v[c] = acc;
                }
                const int m = m0 + p;
                if constexpr (OUT == 2) {
                    const int off = (m * a.y_ldc + a.y_coff + c0) * 4;
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        __builtin_amdgcn_raw_buffer_store_b32(v[c], ry, off + 4 * c, 0, kStream);
                    continue;
                }
                uint32_t packed = 0u;
                if constexpr (OUT == 0) {
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        const int u = (__mulhi(v[c], cr[c].mult) + cr[c].rndzp) >> (cr[c].shift & 31);
                        packed |= (uint32_t)clamp_i32(u, a.lo_off, a.hi_off) << (8 * c);
                    }
                    packed ^= a.out_xor;
                } else {
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        long long o8 = rounding_mul_shift(v[c], cr[c].mult, cr[c].shift, a.rounding) + a.zp_y;
                        o8 = o8 < a.lo ? a.lo : (o8 > a.hi ? a.hi : o8);
                        packed |= ((uint32_t)o8 & 0xffu) << (8 * c);
                    }
                }
                const int off = m * a.y_ldc + a.y_coff + c0;
                if (a.vec_store) {
                    __builtin_amdgcn_raw_buffer_store_b32(packed, ry, off, 0, kStream);
                } else {
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        __builtin_amdgcn_raw_buffer_store_b8((uint8_t)(packed >> (8 * c)), ry, off + c, 0, kStream);
                }
            }
        };

        uint32_t TA[4][P], TB[4][P], TC[4][P];
        if constexpr (SH == 1) {
            // output row o reads input rows o, o + 1, o + 2 of the band
            taps(0, TA);
            taps(1, TB);
            for (int o = 0; o < rows; o += 3) {
                taps(o + 2, TC);
                out_row(o, TA, TB, TC);
                if (o + 1 >= rows)
                    break;
                taps(o + 3, TA);
                out_row(o + 1, TB, TC, TA);
                if (o + 2 >= rows)
                    break;
                taps(o + 4, TB);
                out_row(o + 2, TC, TA, TB);
            }
        } else {
            // output row o reads input rows 2 o, 2 o + 1, 2 o + 2
            taps(0, TA);
            for (int o = 0; o < rows; o += 2) {
                taps(2 * o + 1, TB);
                taps(2 * o + 2, TC);
                out_row(o, TA, TB, TC);
                if (o + 1 >= rows)
                    break;
                taps(2 * o + 3, TB);
                taps(2 * o + 4, TA);
                out_row(o + 1, TC, TB, TA);
            }
        }
    }
}

template <int SW, int SH, bool FLIP, bool ZPW>
static void launch_band_out(const DwArgs &a, dim3 grid, hipStream_t st)
{
    const dim3 block((unsigned)a.bthreads);
    if (a.out_i32)
        launch_main((depthwise3_band_kernel<SW, SH, FLIP, ZPW, 2>), grid, block, (unsigned)a.lbytes, st, a);
    else if (a.fast_rq)
        launch_main((depthwise3_band_kernel<SW, SH, FLIP, ZPW, 0>), grid, block, (unsigned)a.lbytes, st, a);
    else
        launch_main((depthwise3_band_kernel<SW, SH, FLIP, ZPW, 1>), grid, block, (unsigned)a.lbytes, st, a);
}

template <int SW, int SH>
static void launch_band_flags(const DwArgs &a, dim3 grid, hipStream_t st)
{
    const bool flip = a.flip4 != 0;
    if (flip)
        a.zpw_any ? launch_band_out<SW, SH, true, true>(a, grid, st) : launch_band_out<SW, SH, true, false>(a, grid, st);
    else
        a.zpw_any ? launch_band_out<SW, SH, false, true>(a, grid, st)
                  : launch_band_out<SW, SH, false, false>(a, grid, st);
}

hipError_t launch_depthwise3_band(const DwArgs &a, hipStream_t st)
{
    if (!a.band || a.R != 3 || a.S != 3 || a.dh != 1 || a.dw != 1 || a.C % 8 != 0 || (a.W * a.C) % 16 != 0 ||
        (a.sw != 1 && a.sw != 2) || (a.sh != 1 && a.sh != 2) || a.rb < 1 || a.nband < 1 || a.ct < 1 ||
        a.nct < 1 || (a.nct > 1 && a.C % 16 != 0) || a.bthreads < 64 || a.bthreads > 512 || a.bthreads % 64 != 0 ||
        a.lbytes > 65536 || ((uintptr_t)a.x & 15) != 0)
        return hipErrorInvalidValue;
    if ((int64_t)a.N * a.Ho * a.Wo == 0)
        return hipSuccess;
    const unsigned wgs = (unsigned)a.N * (unsigned)a.nband * (unsigned)a.nct;
    const dim3 grid((wgs + 7) / 8 * 8);
    if (a.sw == 1)
        a.sh == 1 ? launch_band_flags<1, 1>(a, grid, st) : launch_band_flags<1, 2>(a, grid, st);
    else
        a.sh == 1 ? launch_band_flags<2, 1>(a, grid, st) : launch_band_flags<2, 2>(a, grid, st);
    return hipGetLastError();
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

template <int SW, int T, bool ZPW, int OUT>
static void launch_dw3_cfg(const DwArgs &a, dim3 grid, hipStream_t st)
{
    launch_main((depthwise3_kernel<SW, kDw3Pixels, T, ZPW, OUT>), grid, dim3(256), 0, st, a);
}

template <int SW, int T, bool ZPW>
static void launch_dw3_out(const DwArgs &a, dim3 grid, hipStream_t st)
{
    if (a.out_i32)
        launch_dw3_cfg<SW, T, ZPW, 2>(a, grid, st);
    else if (a.fast_rq)
        launch_dw3_cfg<SW, T, ZPW, 0>(a, grid, st);
    else
        launch_dw3_cfg<SW, T, ZPW, 1>(a, grid, st);
}

template <int SW, int T>
static void launch_dw3_zpw(const DwArgs &a, dim3 grid, hipStream_t st)
{
    if (a.zpw_any)
        launch_dw3_out<SW, T, true>(a, grid, st);
    else
        launch_dw3_out<SW, T, false>(a, grid, st);
}

template <int SW>
static hipError_t launch_dw3_seg(const DwArgs &a, dim3 grid, hipStream_t st)
{
    switch (a.seg) {
    case 1: launch_dw3_zpw<SW, 1>(a, grid, st); break;
    case 2: launch_dw3_zpw<SW, 2>(a, grid, st); break;
    case 4: launch_dw3_zpw<SW, 4>(a, grid, st); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_depthwise3(const DwArgs &a, hipStream_t st)
{
    if (a.R != 3 || a.S != 3 || a.dh != 1 || a.dw != 1 || a.C % 8 != 0 || a.sh < 1 || (a.sw != 1 && a.sw != 2))
        return hipErrorInvalidValue;
    if (a.items == 0)
        return hipSuccess;
    const dim3 grid((unsigned)(((a.items + 255) / 256 + 7) / 8 * 8));
    return a.sw == 1 ? launch_dw3_seg<1>(a, grid, st) : launch_dw3_seg<2>(a, grid, st);
}

int dw3_pixels()
{
    return kDw3Pixels;
}

}  // namespace qnn
