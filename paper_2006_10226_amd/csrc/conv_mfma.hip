// Implicit-GEMM quantized conv2d / dense on gfx950 int8 MFMA with a fused
// zero-point + requantize epilogue.
//
// Method (Jain et al., Sec. II-B Eq. (3), Sec. III-B/C):
//   acc[m,k] = sum_j (x~[m,j] - zp_x)(w[k,j] - zp_w[k])
//            = sum_j x~'[m,j] w[k,j]                    (term 1: the MFMA GEMM)
//              - zp_x' * sum_j w[k,j]                    (term 2, folded at plan time)
//              - zp_w[k] * sum_j x~'[m,j]                (term 3, only if zp_w != 0)
//              + J * zp_x' * zp_w[k]                     (term 4, folded at plan time)
// where x' = x - 128 with zp_x' = zp_x - 128 when x is uint8 (the
// legalisation of Sec. III-C: the int8 MFMA is signed x signed, and the
// shift leaves every (x - zp_x) unchanged) and x~ holds zp_x at padded taps.
// Terms 2 and 4 plus the bias are one per-channel constant (ChanRec.bconst).
//
// GEMM orientation: the MFMA "A" operand is the weight tile (rows = output
// channels), "B" is the gathered activation tile (columns = output pixels),
// so each lane of a v_mfma_i32_16x16x64_i8 result holds 4 consecutive
// output channels of one pixel: the epilogue stores 4 bytes at once into the
// NHWC output.  Tiles are staged through LDS with an XOR swizzle of the
// 16-byte chunks, double buffered, one barrier per K-step.
#include "qnn_internal.h"

namespace qnn {

typedef int v4i __attribute__((ext_vector_type(4)));

TileShape tile_shape(int tile)
{
    switch (tile) {
    case TILE_128x128: return {128, 128, 128};
    case TILE_64x256: return {64, 256, 128};
    case TILE_256x128: return {256, 128, 128};
    default: return {64, 64, 128};
    }
}

int gather_width(int C)
{
    if (C % 16 == 0) return 16;
    if (C % 4 == 0) return 4;
    return 1;
}

// Physical 16-byte chunk of logical chunk q in LDS row `row` (rows of BK
// bytes).  A 16-lane group reading rows 0..15 at one logical chunk touches
// 16 distinct 16-byte bank groups, and each 8-lane half touches 8.
template <int CPR>
__device__ __forceinline__ int swizzle(int row)
{
    static_assert(CPR == 8 || CPR == 4, "BK must be 64 or 128");
    if constexpr (CPR == 8)
        return (row & 7) ^ ((row >> 3) & 1);
    else
        return ((row >> 1) & 3) ^ ((row >> 3) & 1);
}

// Fixed-point requantize of v: round(v * mult / 2^shift) with the selected
// rounding, as a 64-bit product (|v| <= 2^31, mult < 2^31).
__device__ __forceinline__ long long round_mul_shift(int v, int mult, int shift, int rounding)
{
    long long p = (long long)v * (long long)mult;
    long long half = 1LL << (shift - 1);
    if (rounding == 0)
        return (p + half) >> shift;
    long long a = p < 0 ? -p : p;
    long long t = (a + half) >> shift;
    return p < 0 ? -t : t;
}

__device__ __forceinline__ int clamp_i(long long v, int lo, int hi)
{
    return (int)(v < lo ? lo : (v > hi ? hi : v));
}

// Map a workgroup id onto a tile so that consecutive tiles (which share an
// activation tile across channel tiles) land on the same XCD: workgroups
// are dispatched round-robin over the 8 XCDs.
__device__ __forceinline__ int xcd_remap(int bid, int nblocks)
{
    const int q = nblocks >> 3, r = nblocks & 7;
    const int x = bid & 7, i = bid >> 3;
    return x * q + (x < r ? x : r) + i;
}

// Two workgroups per CU (2 waves per SIMD) when both double-buffered tiles fit
// twice into the 160 KB LDS, else one.
template <int TC, int TP, int BK, int WC, int WP, int AVEC, int MODE, bool TERM3>
__global__ void __launch_bounds__(256, ((TC + TP) * BK * 2 <= 80 * 1024) ? 2 : 1) conv_mfma_kernel(ConvArgs a)
{
    constexpr int NT = 256;
    constexpr int CPR = BK / 16;                // 16-byte chunks per LDS row
    constexpr int RPP = NT / CPR;               // rows loaded per pass of the block
    constexpr int A_PASS = TC / RPP;            // weight rows per thread
    constexpr int B_PASS = TP / RPP;            // pixel rows per thread
    constexpr int WTC = TC / WC, WTP = TP / WP; // wave tile
    constexpr int FC = WTC / 16, FP = WTP / 16; // 16x16 MFMA blocks per wave
    static_assert(WC * WP == 4, "4 waves per workgroup");
    static_assert(TC % RPP == 0 && TP % RPP == 0, "tile rows must fill the passes");
    static_assert(AVEC == 16 || AVEC == 4 || AVEC == 1, "gather width");

    __shared__ __attribute__((aligned(16))) int8_t lds[2][(TC + TP) * BK];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wc = wave / WP, wpos = wave % WP;

    const int tile = xcd_remap(blockIdx.x, a.nblocks);
    const int c0 = (tile % a.tiles_c) * TC;
    const int p0 = (tile / a.tiles_c) * TP;
    const int split = blockIdx.y;
    const int nk_total = a.Jpad / BK;
    const int k_begin = split * a.ksteps;
    const int k_end = min(nk_total, k_begin + a.ksteps);

    // ---- loader state --------------------------------------------------
    const int q = tid % CPR;      // chunk column this thread loads
    const int rbase = tid / CPR;  // first row this thread loads

    // activation pixel rows
    int pix_base[B_PASS], ih0[B_PASS], iw0[B_PASS];
    bool pvalid[B_PASS];
#pragma unroll
    for (int i = 0; i < B_PASS; ++i) {
        const int m = p0 + rbase + i * RPP;
        pvalid[i] = m < a.M;
        const int mm = pvalid[i] ? m : 0;
        const int ow = mm % a.Wo;
        const int t = mm / a.Wo;
        const int oh = t % a.Ho;
        const int n = t / a.Ho;
        pix_base[i] = n * a.H * a.W * a.C;
        ih0[i] = oh * a.sh - a.pt;
        iw0[i] = ow * a.sw - a.pl;
    }

    // (r, s, c) of this thread's chunk at the current K-step (16-byte gather)
    int gr = 0, gs = 0, gc = 0;
    if constexpr (AVEC == 16) {
        const int j0 = k_begin * BK + q * 16;
        const int t = j0 / a.C;
        gc = j0 - t * a.C;
        gs = t % a.S;
        gr = t / a.S;
    }

    const int8_t *wrow = a.wp + (size_t)(c0 + rbase) * a.Jpad + q * 16;

    int4 ra[A_PASS], rb[B_PASS];

    auto load_tile = [&](int kt) {
#pragma unroll
        for (int i = 0; i < A_PASS; ++i)
            ra[i] = *(const int4 *)(wrow + (size_t)i * RPP * a.Jpad + (size_t)kt * BK);
        if constexpr (AVEC == 16) {
            const bool kin = gr < a.R;
            const int dr = gr * a.dh, ds = gs * a.dw;
#pragma unroll
            for (int i = 0; i < B_PASS; ++i) {
                const int ih = ih0[i] + dr, iw = iw0[i] + ds;
                int4 v;
                if (pvalid[i] && kin) {
                    if ((unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W) {
                        v = *(const int4 *)(a.x + pix_base[i] + (ih * a.W + iw) * a.C + gc);
                        v.x ^= a.flip4; v.y ^= a.flip4; v.z ^= a.flip4; v.w ^= a.flip4;
                    } else {
                        v = make_int4(a.pad4, a.pad4, a.pad4, a.pad4);
                    }
                } else {
                    v = make_int4(0, 0, 0, 0);
                }
                rb[i] = v;
            }
        } else {
            // narrow gather: pieces of AVEC bytes, each inside one filter tap
            const int jb = kt * BK + q * 16;
#pragma unroll
            for (int i = 0; i < B_PASS; ++i) {
                uint32_t words[4] = {0, 0, 0, 0};
#pragma unroll
                for (int pc = 0; pc < 16 / AVEC; ++pc) {
                    const int j = jb + pc * AVEC;
                    uint32_t piece = 0;
                    if (pvalid[i] && j < a.J) {
                        const int t = j / a.C;
                        const int c = j - t * a.C;
                        const int s = t % a.S, r = t / a.S;
                        const int ih = ih0[i] + r * a.dh, iw = iw0[i] + s * a.dw;
                        if ((unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W) {
                            const uint8_t *src = a.x + pix_base[i] + (ih * a.W + iw) * a.C + c;
                            if constexpr (AVEC == 4)
                                piece = *(const uint32_t *)src ^ a.flip4;
                            else
                                piece = (uint32_t)(*src) ^ (a.flip4 & 0xffu);
                        } else {
                            piece = AVEC == 4 ? a.pad4 : (a.pad4 & 0xffu);
                        }
                    }
                    if constexpr (AVEC == 4)
                        words[pc] = piece;
                    else
                        words[pc >> 2] |= piece << (8 * (pc & 3));
                }
                rb[i] = make_int4(words[0], words[1], words[2], words[3]);
            }
        }
    };

    auto advance = [&]() {
        if constexpr (AVEC == 16) {
            gc += BK;
            while (gc >= a.C) {
                gc -= a.C;
                if (++gs == a.S) {
                    gs = 0;
                    ++gr;
                }
            }
        }
    };

    auto store_tile = [&](int buf) {
        int8_t *As = lds[buf];
        int8_t *Bs = lds[buf] + TC * BK;
#pragma unroll
        for (int i = 0; i < A_PASS; ++i) {
            const int row = rbase + i * RPP;
            *(int4 *)(As + row * BK + ((q ^ swizzle<CPR>(row)) << 4)) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < B_PASS; ++i) {
            const int row = rbase + i * RPP;
            *(int4 *)(Bs + row * BK + ((q ^ swizzle<CPR>(row)) << 4)) = rb[i];
        }
    };

    v4i acc[FC][FP];
#pragma unroll
    for (int i = 0; i < FC; ++i)
#pragma unroll
        for (int jj = 0; jj < FP; ++jj)
            acc[i][jj] = v4i{0, 0, 0, 0};

    if (k_begin < k_end) {
        load_tile(k_begin);
        store_tile(0);
    }
    __syncthreads();

    const int lrow = lane & 15;   // operand row inside a 16x16 block
    const int lchk = lane >> 4;   // 16-byte k-chunk inside a 64-wide k slice

    for (int kt = k_begin; kt < k_end; ++kt) {
        const int buf = (kt - k_begin) & 1;
        const bool more = kt + 1 < k_end;
        if (more) {
            advance();
            load_tile(kt + 1);
        }
        const int8_t *As = lds[buf];
        const int8_t *Bs = lds[buf] + TC * BK;
#pragma unroll
        for (int kk = 0; kk < BK / 64; ++kk) {
            const int chunk = kk * 4 + lchk;
            v4i fa[FC], fb[FP];
#pragma unroll
            for (int i = 0; i < FC; ++i) {
                const int row = wc * WTC + i * 16 + lrow;
                fa[i] = *(const v4i *)(As + row * BK + ((chunk ^ swizzle<CPR>(row)) << 4));
            }
#pragma unroll
            for (int jj = 0; jj < FP; ++jj) {
                const int row = wpos * WTP + jj * 16 + lrow;
                fb[jj] = *(const v4i *)(Bs + row * BK + ((chunk ^ swizzle<CPR>(row)) << 4));
            }
#pragma unroll
            for (int i = 0; i < FC; ++i)
#pragma unroll
                for (int jj = 0; jj < FP; ++jj)
                    acc[i][jj] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[jj], acc[i][jj], 0, 0, 0);
        }
        if (more)
            store_tile(buf ^ 1);
        __syncthreads();
    }

    // ---- epilogue --------------------------------------------------------
    // lane holds channels ch..ch+3 (4 * (lane >> 4) inside the 16-block) of
    // pixel m (lane & 15 inside the 16-block).
#pragma unroll
    for (int i = 0; i < FC; ++i) {
        const int ch = c0 + wc * WTC + i * 16 + lchk * 4;
        if (ch >= a.K)
            continue;
        int mult[4], shift[4], bconst[4], zpw[4];
        if constexpr (MODE != OUT_PARTIAL) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const ChanRec cr = a.chan[ch + e];
                mult[e] = cr.mult; shift[e] = cr.shift; bconst[e] = cr.bconst; zpw[e] = cr.zpw;
            }
        }
#pragma unroll
        for (int jj = 0; jj < FP; ++jj) {
            const int m = p0 + wpos * WTP + jj * 16 + lrow;
            if (m >= a.M)
                continue;
            if constexpr (MODE == OUT_PARTIAL) {
                int32_t *dst = a.ws + ((size_t)split * a.M + m) * a.Kpad + ch;
                *(v4i *)dst = acc[i][jj];
                continue;
            } else {
                int vals[4];
                const int asum = TERM3 ? a.asum[m] : 0;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    // wrap-around int32 arithmetic; exact when the true value fits
                    uint32_t v = (uint32_t)acc[i][jj][e] + (uint32_t)bconst[e];
                    if (TERM3)
                        v -= (uint32_t)zpw[e] * (uint32_t)asum;
                    vals[e] = (int)v;
                }
                const size_t off = (size_t)m * a.y_ldc + a.y_coff + ch;
                if constexpr (MODE == OUT_INT32) {
                    int32_t *yp = (int32_t *)a.y + off;
                    if (a.vec_store && ch + 3 < a.K) {
                        *(int4 *)yp = make_int4(vals[0], vals[1], vals[2], vals[3]);
                    } else {
                        for (int e = 0; e < 4 && ch + e < a.K; ++e)
                            yp[e] = vals[e];
                    }
                } else {
                    uint32_t packed = 0;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const long long t = round_mul_shift(vals[e], mult[e], shift[e], a.rounding);
                        const int o = clamp_i(t + a.zp_y, a.lo, a.hi);
                        packed |= ((uint32_t)o & 0xffu) << (8 * e);
                    }
                    uint8_t *yp = (uint8_t *)a.y + off;
                    if (a.vec_store && ch + 3 < a.K) {
                        *(uint32_t *)yp = packed;
                    } else {
                        for (int e = 0; e < 4 && ch + e < a.K; ++e)
                            yp[e] = (uint8_t)(packed >> (8 * e));
                    }
                }
            }
        }
    }
}

// Sum the split-K partials of (pixel m, channels 4g..4g+3) and apply the
// same epilogue as the fused kernel.
template <int MODE, bool TERM3>
__global__ void __launch_bounds__(256) splitk_reduce_kernel(ConvArgs a)
{
    const int groups = a.Kpad / 4;
    const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= (long long)a.M * groups)
        return;
    const int m = (int)(gid / groups);
    const int ch = (int)(gid % groups) * 4;
    if (ch >= a.K)
        return;
    uint32_t acc[4] = {0, 0, 0, 0};
    for (int s = 0; s < a.nsplit; ++s) {
        const int4 p = *(const int4 *)(a.ws + ((size_t)s * a.M + m) * a.Kpad + ch);
        acc[0] += (uint32_t)p.x; acc[1] += (uint32_t)p.y;
        acc[2] += (uint32_t)p.z; acc[3] += (uint32_t)p.w;
    }
    const int asum = TERM3 ? a.asum[m] : 0;
    int vals[4];
    for (int e = 0; e < 4; ++e) {
        const ChanRec cr = a.chan[ch + e];
        uint32_t v = acc[e] + (uint32_t)cr.bconst;
        if (TERM3)
            v -= (uint32_t)cr.zpw * (uint32_t)asum;
        vals[e] = (int)v;
    }
    const size_t off = (size_t)m * a.y_ldc + a.y_coff + ch;
    if constexpr (MODE == OUT_INT32) {
        int32_t *yp = (int32_t *)a.y + off;
        for (int e = 0; e < 4 && ch + e < a.K; ++e)
            yp[e] = vals[e];
    } else {
        uint8_t *yp = (uint8_t *)a.y + off;
        for (int e = 0; e < 4 && ch + e < a.K; ++e) {
            const ChanRec cr = a.chan[ch + e];
            const long long t = round_mul_shift(vals[e], cr.mult, cr.shift, a.rounding);
            yp[e] = (uint8_t)clamp_i(t + a.zp_y, a.lo, a.hi);
        }
    }
}

// Term 3 of Eq. (3): asum[m] = sum over the receptive field of x~' (the
// legalised input, zp_x' at padded taps).  Only needed when some zp_w != 0.
__global__ void __launch_bounds__(256) window_sum_kernel(ConvArgs a, int32_t *out)
{
    const int m = blockIdx.x * blockDim.x + threadIdx.x;
    if (m >= a.M)
        return;
    const int ow = m % a.Wo, t = m / a.Wo, oh = t % a.Ho, n = t / a.Ho;
    const int pad = (int)(int8_t)(a.pad4 & 0xffu);
    const int flip = (int)(a.flip4 & 0xffu);
    int sum = 0;
    for (int r = 0; r < a.R; ++r)
        for (int s = 0; s < a.S; ++s) {
            const int ih = oh * a.sh - a.pt + r * a.dh, iw = ow * a.sw - a.pl + s * a.dw;
            if ((unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W) {
                const uint8_t *src = a.x + ((size_t)(n * a.H + ih) * a.W + iw) * a.C;
                for (int c = 0; c < a.C; ++c)
                    sum += (int)(int8_t)(uint8_t)(src[c] ^ flip);
            } else {
                sum += pad * a.C;
            }
        }
    out[m] = sum;
}

// Plan preparation: pack w[K][J] into [Kpad][Jpad] (zero padded) and fold
// bias, term 2 and term 4 into chan[k].bconst.  chan[k].mult/shift/zpw were
// uploaded by the host.  One workgroup per (padded) output channel.
__global__ void __launch_bounds__(256) prep_conv_kernel(const int8_t *w, const int32_t *bias, int K,
                                                        int J, int Jpad, int32_t zpx, int8_t *wp,
                                                        ChanRec *chan)
{
    const int k = blockIdx.x;
    __shared__ long long part[256];
    long long sum = 0;
    for (int j = threadIdx.x; j < Jpad; j += blockDim.x) {
        int8_t v = 0;
        if (k < K && j < J)
            v = w[(size_t)k * J + j];
        wp[(size_t)k * Jpad + j] = v;
        sum += v;
    }
    part[threadIdx.x] = sum;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off)
            part[threadIdx.x] += part[threadIdx.x + off];
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        if (k < K) {
            const long long wsum = part[0];
            const long long zpw = chan[k].zpw;
            const long long b = bias ? (long long)bias[k] : 0;
            const long long c = b - (long long)zpx * wsum + (long long)J * zpx * zpw;
            chan[k].bconst = (int32_t)(uint32_t)(unsigned long long)c;
        } else {
            chan[k] = ChanRec{0, 1, 0, 0};
        }
    }
}

template <int TC, int TP, int BK, int WC, int WP, int AVEC>
static hipError_t launch_cfg(const ConvArgs &a, int mode, hipStream_t st)
{
    dim3 grid(a.nblocks, a.nsplit), block(256);
    const bool t3 = a.asum != nullptr;
    if (mode == OUT_PARTIAL) {
        hipLaunchKernelGGL((conv_mfma_kernel<TC, TP, BK, WC, WP, AVEC, OUT_PARTIAL, false>), grid, block, 0, st, a);
    } else if (mode == OUT_INT32) {
        if (t3)
            hipLaunchKernelGGL((conv_mfma_kernel<TC, TP, BK, WC, WP, AVEC, OUT_INT32, true>), grid, block, 0, st, a);
        else
            hipLaunchKernelGGL((conv_mfma_kernel<TC, TP, BK, WC, WP, AVEC, OUT_INT32, false>), grid, block, 0, st, a);
    } else {
        if (t3)
            hipLaunchKernelGGL((conv_mfma_kernel<TC, TP, BK, WC, WP, AVEC, OUT_REQUANT, true>), grid, block, 0, st, a);
        else
            hipLaunchKernelGGL((conv_mfma_kernel<TC, TP, BK, WC, WP, AVEC, OUT_REQUANT, false>), grid, block, 0, st, a);
    }
    return hipGetLastError();
}

template <int TC, int TP, int BK, int WC, int WP>
static hipError_t launch_avec(const ConvArgs &a, int avec, int mode, hipStream_t st)
{
    if (avec == 16) return launch_cfg<TC, TP, BK, WC, WP, 16>(a, mode, st);
    if (avec == 4) return launch_cfg<TC, TP, BK, WC, WP, 4>(a, mode, st);
    return launch_cfg<TC, TP, BK, WC, WP, 1>(a, mode, st);
}

hipError_t launch_conv(const ConvArgs &a, int tile, int avec, int mode, hipStream_t st)
{
    switch (tile) {
    case TILE_128x128: return launch_avec<128, 128, 128, 2, 2>(a, avec, mode, st);
    case TILE_64x256: return launch_avec<64, 256, 128, 1, 4>(a, avec, mode, st);
    case TILE_256x128: return launch_avec<256, 128, 128, 2, 2>(a, avec, mode, st);
    default: return launch_avec<64, 64, 128, 2, 2>(a, avec, mode, st);
    }
}

hipError_t launch_splitk_reduce(const ConvArgs &a, int mode, hipStream_t st)
{
    const long long n = (long long)a.M * (a.Kpad / 4);
    dim3 grid((unsigned)((n + 255) / 256)), block(256);
    const bool t3 = a.asum != nullptr;
    if (mode == OUT_INT32) {
        if (t3) hipLaunchKernelGGL((splitk_reduce_kernel<OUT_INT32, true>), grid, block, 0, st, a);
        else hipLaunchKernelGGL((splitk_reduce_kernel<OUT_INT32, false>), grid, block, 0, st, a);
    } else {
        if (t3) hipLaunchKernelGGL((splitk_reduce_kernel<OUT_REQUANT, true>), grid, block, 0, st, a);
        else hipLaunchKernelGGL((splitk_reduce_kernel<OUT_REQUANT, false>), grid, block, 0, st, a);
    }
    return hipGetLastError();
}

hipError_t launch_window_sums(const ConvArgs &a, int32_t *out, hipStream_t st)
{
    dim3 grid((a.M + 255) / 256), block(256);
    hipLaunchKernelGGL(window_sum_kernel, grid, block, 0, st, a, out);
    return hipGetLastError();
}

hipError_t launch_prep_conv(const int8_t *w, const int32_t *bias, int K, int J, int Jpad, int Kpad,
                            int32_t zpx, int8_t *wp, ChanRec *chan, hipStream_t st)
{
    hipLaunchKernelGGL(prep_conv_kernel, dim3(Kpad), dim3(256), 0, st, w, bias, K, J, Jpad, zpx, wp, chan);
    return hipGetLastError();
}

}  // namespace qnn
