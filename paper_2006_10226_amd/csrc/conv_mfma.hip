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
typedef int v2i __attribute__((ext_vector_type(2)));

TileShape tile_shape(int tile)
{
    switch (tile) {
    case TILE_128x128: return {128, 128, 128};
    case TILE_64x256: return {64, 256, 128};
    case TILE_256x128: return {256, 128, 128};
    case TILE_64x64: return {64, 64, 128};
    case TILE_64x64_K64: return {64, 64, 64};
    case TILE_128x128_K64: return {128, 128, 64};
    case TILE_128x64: return {128, 64, 128};
    case TILE_256x64_K64: return {256, 64, 64};
    default: return {64, 128, 128};
    }
}

int gather_width(int C)
{
    if (C % 16 == 0) return 16;
    if (C % 8 == 0) return 8;
    return 4;  // C % 4 == 0 (other channel counts are padded to a multiple of 4)
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

// The 32-bit form used by the conv epilogue when rounding is HALF_UP and
// 33 <= shift <= 53: with hi = floor(v*mult / 2^32) (the signed high word of
// the product) and sh = shift - 32,
//   floor((v*mult + 2^(shift-1)) / 2^shift) = floor((hi + 2^(sh-1)) / 2^sh),
// because the low word only adds a fraction below 1 before the integer
// division by 2^sh; adding (zp + off) * 2^sh before the shift adds exactly
// zp + off after it.  |hi| <= 2^30 and (zp + off) * 2^sh <= 255 * 2^21, so
// the 32-bit sum cannot overflow.

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

// Four consecutive channel records, from the LDS copy when there is one
// (explicit LDS reads keep them off the vector-memory counter) or from
// global memory.
__device__ __forceinline__ void load_chan4(bool in_lds, const ChanRec *lds_tab, const ChanRec *g_tab, int c,
                                           int mult[4], int bconst[4], int rndzp[4], int shift[4])
{
    if (in_lds) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const v4i cr = *(const __attribute__((address_space(3))) v4i *)(
                (const __attribute__((address_space(3))) ChanRec *)lds_tab + c + e);
            mult[e] = cr.x; bconst[e] = cr.y; rndzp[e] = cr.z; shift[e] = cr.w;
        }
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const v4i cr = *(const v4i *)(g_tab + c + e);
            mult[e] = cr.x; bconst[e] = cr.y; rndzp[e] = cr.z; shift[e] = cr.w;
        }
    }
}

// Load of AVEC bytes (16, 8 or 4) as 4, 2 or 1 dwords.
template <int AVEC>
struct Piece;
template <>
struct Piece<16> {
    v4i v;
    __device__ __forceinline__ void load(const uint8_t *p) { v = *(const v4i *)p; }
};
template <>
struct Piece<8> {
    v2i v;
    __device__ __forceinline__ void load(const uint8_t *p) { v = *(const v2i *)p; }
};
template <>
struct Piece<4> {
    int v;
    __device__ __forceinline__ void load(const uint8_t *p) { v = *(const int *)p; }
};

// Persistent implicit-GEMM kernel.  Each workgroup walks a list of output
// tiles (TC channels x TP pixels); the K-steps of all its tiles form one
// stream of stages.  A ring of D register stages keeps the global loads of
// the next D-1 stages in flight -- across tile boundaries, so the next
// tile's loads overlap this tile's epilogue -- and two LDS buffers feed the
// MFMAs.  Gathers of padded taps, of the K tail and of rows past M read a
// 16-byte device buffer holding zp_x instead of branching: for padded taps
// that is exactly the value the paper pads with, and the other two are
// multiplied by zero weights or discarded.
template <int TC, int TP, int BK, int WC, int WP, int AVEC, int D>
__global__ void __launch_bounds__(256, ((TC + TP) * BK * 2 <= 80 * 1024) ? 2 : 1) conv_mfma_kernel(ConvArgs a)
{
    constexpr int NT = 256;
    constexpr int CPR = BK / 16;                // 16-byte chunks per LDS row
    constexpr int RPP = NT / CPR;               // rows loaded per pass of the block
    constexpr int A_PASS = TC / RPP;            // weight rows per thread
    constexpr int B_PASS = TP / RPP;            // pixel rows per thread
    constexpr int WTC = TC / WC, WTP = TP / WP; // wave tile
    constexpr int FC = WTC / 16, FP = WTP / 16; // 16x16 MFMA blocks per wave
    constexpr int NPC = 16 / AVEC;              // gather pieces per 16-byte chunk
    static_assert(WC * WP == 4, "4 waves per workgroup");
    static_assert(TC % RPP == 0 && TP % RPP == 0, "tile rows must fill the passes");
    static_assert(AVEC == 16 || AVEC == 8 || AVEC == 4, "gather width");
    static_assert(D % 2 == 0 && D >= 2, "ring depth must be even");

    __shared__ __attribute__((aligned(16))) int8_t lds[2][(TC + TP) * BK];
    // per-channel epilogue records, copied once per workgroup: reading them
    // from LDS keeps the epilogue off the in-order vector-memory counter,
    // which would otherwise drain the whole prefetch ring at every tile end
    extern __shared__ __attribute__((aligned(16))) int8_t dyn_lds[];
    ChanRec *chan_lds = (ChanRec *)dyn_lds;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wc = wave / WP, wpos = wave % WP;

    // ---- work assignment: XCD x (workgroups x, x+8, ...) owns the x-th
    // eighth of the tile range, so tiles that share activations (consecutive
    // ids: all channel tiles of a pixel tile) share that XCD's L2.
    const int xcd = blockIdx.x & 7, lb = blockIdx.x >> 3;
    const int gx = gridDim.x >> 3;
    const int chunk = (a.ntiles + 7) >> 3;
    const int t_first = xcd * chunk + lb;
    const int t_end = min(a.ntiles, (xcd + 1) * chunk);
    const int my_tiles = t_first < t_end ? (t_end - t_first + gx - 1) / gx : 0;
    const int nk = a.nk;
    const int G = my_tiles * nk;
    if (G == 0)
        return;
    if (a.chan_in_lds) {
        for (int i = tid; i < a.Kpad; i += NT)
            *(v4i *)(chan_lds + i) = *(const v4i *)(a.chan + i);
        // made visible by the barrier after the prologue's first LDS store
    }

    // ---- loader (runs up to D-1 stages ahead of the MFMAs) ---------------
    const int q = tid % CPR;      // chunk column this thread loads
    const int rbase = tid / CPR;  // first row this thread loads

    int l_tile = 0, l_k = 0;      // loader position: tile ordinal, K-step
    int pix_base[B_PASS], ih0[B_PASS], iw0[B_PASS];
    bool pvalid[B_PASS];
    int gr[NPC], gs[NPC], gc[NPC], gr0[NPC], gs0[NPC], gc0[NPC];
#pragma unroll
    for (int pc = 0; pc < NPC; ++pc) {
        const int j0 = q * 16 + pc * AVEC;
        const int t = j0 / a.C;
        gc0[pc] = j0 - t * a.C;
        gs0[pc] = t % a.S;
        gr0[pc] = t / a.S;
    }
    const int dtap = BK / a.C, dc = BK - dtap * a.C;
    const int dts = dtap % a.S, dtr = dtap / a.S;
    const int8_t *wrow = a.wp;

    auto begin_tile = [&](int ordinal) {
        const int tile = t_first + ordinal * gx;
        const int c0 = (tile % a.tiles_c) * TC;
        const int p0 = (tile / a.tiles_c) * TP;
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
#pragma unroll
        for (int pc = 0; pc < NPC; ++pc) {
            gr[pc] = gr0[pc];
            gs[pc] = gs0[pc];
            gc[pc] = gc0[pc];
        }
        wrow = a.wp + (size_t)(c0 + rbase) * a.Jpad + q * 16;
    };

    auto next_stage = [&]() {
        if (++l_k == nk) {
            l_k = 0;
            if (++l_tile < my_tiles)
                begin_tile(l_tile);
            return;
        }
#pragma unroll
        for (int pc = 0; pc < NPC; ++pc) {
            gc[pc] += dc;
            int carry = gc[pc] >= a.C;
            gc[pc] -= carry ? a.C : 0;
            gs[pc] += dts + carry;
            carry = gs[pc] >= a.S;
            gs[pc] -= carry ? a.S : 0;
            gr[pc] += dtr + carry;
        }
    };

    v4i ra[D][A_PASS];
    Piece<AVEC> rb[D][B_PASS][NPC];

    auto load_stage = [&](v4i (&A)[A_PASS], Piece<AVEC> (&B)[B_PASS][NPC]) {
#pragma unroll
        for (int i = 0; i < A_PASS; ++i)
            A[i] = *(const v4i *)(wrow + (size_t)i * RPP * a.Jpad + (size_t)l_k * BK);
#pragma unroll
        for (int pc = 0; pc < NPC; ++pc) {
            const bool kin = gr[pc] < a.R;
            const int dr = gr[pc] * a.dh, ds = gs[pc] * a.dw;
#pragma unroll
            for (int i = 0; i < B_PASS; ++i) {
                const int ih = ih0[i] + dr, iw = iw0[i] + ds;
                const bool use = pvalid[i] && kin && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
                const uint8_t *src = use ? a.x + pix_base[i] + (ih * a.W + iw) * a.C + gc[pc] : a.padbuf;
                B[i][pc].load(src);
            }
        }
    };

    auto store_stage = [&](int buf, const v4i (&A)[A_PASS], const Piece<AVEC> (&B)[B_PASS][NPC]) {
        int8_t *As = lds[buf];
        int8_t *Bs = lds[buf] + TC * BK;
        const int f = (int)a.flip4;
#pragma unroll
        for (int i = 0; i < A_PASS; ++i) {
            const int row = rbase + i * RPP;
            *(v4i *)(As + row * BK + ((q ^ swizzle<CPR>(row)) << 4)) = A[i];
        }
#pragma unroll
        for (int i = 0; i < B_PASS; ++i) {
            v4i v;
            if constexpr (AVEC == 16)
                v = B[i][0].v;
            else if constexpr (AVEC == 8)
                v = v4i{B[i][0].v.x, B[i][0].v.y, B[i][1].v.x, B[i][1].v.y};
            else
                v = v4i{B[i][0].v, B[i][1].v, B[i][2].v, B[i][3].v};
            v ^= v4i{f, f, f, f};   // uint8 -> int8 legalisation (no-op for int8 input)
            const int row = rbase + i * RPP;
            *(v4i *)(Bs + row * BK + ((q ^ swizzle<CPR>(row)) << 4)) = v;
        }
    };

    v4i acc[FC][FP];
#pragma unroll
    for (int i = 0; i < FC; ++i)
#pragma unroll
        for (int jj = 0; jj < FP; ++jj)
            acc[i][jj] = v4i{0, 0, 0, 0};

    // ---- epilogue of one tile ------------------------------------------
    // lane holds channels ch..ch+3 (4 * (lane >> 4) inside the 16-block) of
    // pixel m (lane & 15 inside the 16-block).  The output mode, term 3 and
    // the requantize form are uniform across the launch (no divergence).
    const int lrow = lane & 15;   // operand row inside a 16x16 block
    const int lchk = lane >> 4;   // 16-byte k-chunk inside a 64-wide k slice
    auto epilogue = [&](int ordinal) {
        const int tile = t_first + ordinal * gx;
        const int c0 = (tile % a.tiles_c) * TC;
        const int p0 = (tile / a.tiles_c) * TP;
        const int mbase = p0 + wpos * WTP + lrow;
        if (a.asum) {
            // term 3 of Eq. (3): - zp_w[k] * (window sum of x~' at pixel m)
#pragma unroll
            for (int i = 0; i < FC; ++i) {
                const int ch = c0 + wc * WTC + i * 16 + lchk * 4;
                const v4i zw = *(const v4i *)(a.zpw + ch);
#pragma unroll
                for (int jj = 0; jj < FP; ++jj) {
                    const int m = min(mbase + jj * 16, a.M - 1);
                    const int s3 = a.asum[m];
                    acc[i][jj] -= zw * v4i{s3, s3, s3, s3};
                }
            }
        }
#pragma unroll
        for (int i = 0; i < FC; ++i) {
            const int ch = c0 + wc * WTC + i * 16 + lchk * 4;
            if (ch >= a.K)
                continue;
            const bool full = a.vec_store && ch + 3 < a.K;
            int mult[4], bconst[4], rndzp[4], shift[4];
            load_chan4(a.chan_in_lds, chan_lds, a.chan, ch, mult, bconst, rndzp, shift);
#pragma unroll
            for (int jj = 0; jj < FP; ++jj) {
                const int m = mbase + jj * 16;
                if (m >= a.M)
                    continue;
                int vals[4];
#pragma unroll
                for (int e = 0; e < 4; ++e)   // wrap-around int32: exact when the true value fits
                    vals[e] = (int)((uint32_t)acc[i][jj][e] + (uint32_t)bconst[e]);
                const size_t off = (size_t)m * a.y_ldc + a.y_coff + ch;
                if (a.mode == OUT_INT32) {
                    int32_t *yp = (int32_t *)a.y + off;
                    if (full) {
                        *(v4i *)yp = v4i{vals[0], vals[1], vals[2], vals[3]};
                    } else {
                        for (int e = 0; e < 4 && ch + e < a.K; ++e)
                            yp[e] = vals[e];
                    }
                    continue;
                }
                uint32_t packed;
                if (a.fast_rq) {
                    // 32-bit requantize; outputs offset into [0, 255] then one XOR
                    // turns the int8 case back into two's complement bytes
                    uint32_t u[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int hi = __mulhi(vals[e], mult[e]);
                        const int t = (hi + rndzp[e]) >> (shift[e] & 31);   // shift - 32 for shift in [33, 53]
                        u[e] = (uint32_t)clamp_i32(t, a.lo_off, a.hi_off);
                    }
                    packed = (u[0] | (u[1] << 8) | (u[2] << 16) | (u[3] << 24)) ^ a.out_xor;
                } else {
                    packed = 0;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int o = clamp_i(rounding_mul_shift(vals[e], mult[e], shift[e], a.rounding) + a.zp_y, a.lo,
                                              a.hi);
                        packed |= ((uint32_t)o & 0xffu) << (8 * e);
                    }
                }
                uint8_t *yp = (uint8_t *)a.y + off;
                if (full) {
                    __builtin_nontemporal_store(packed, (uint32_t *)yp);
                } else {
                    for (int e = 0; e < 4 && ch + e < a.K; ++e)
                        yp[e] = (uint8_t)(packed >> (8 * e));
                }
            }
        }
#pragma unroll
        for (int i = 0; i < FC; ++i)
#pragma unroll
            for (int jj = 0; jj < FP; ++jj)
                acc[i][jj] = v4i{0, 0, 0, 0};
    };

    // Output staged through LDS for whole-row stores: the requantized bytes
    // of the tile are written to `stage` as [TP][SP] with SP = TC + 16 where
    // it fits (the pad spreads the 16 pixel rows of a 4-byte write over
    // more banks), then every thread copies 16-byte chunks of complete pixel
    // rows to y, so a pixel's TC channels leave in one contiguous run.
    constexpr int SP = (TP * (TC + 16) <= (TC + TP) * BK) ? TC + 16 : TC;
    static_assert(TP * SP <= (TC + TP) * BK, "staging must fit one LDS stage buffer");
    auto epilogue_staged = [&](int ordinal, int8_t *stage) {
        const int tile = t_first + ordinal * gx;
        const int c0 = (tile % a.tiles_c) * TC;
        const int p0 = (tile / a.tiles_c) * TP;
        const int mbase = p0 + wpos * WTP + lrow;
        if (a.asum) {
#pragma unroll
            for (int i = 0; i < FC; ++i) {
                const int ch = c0 + wc * WTC + i * 16 + lchk * 4;
                const v4i zw = *(const v4i *)(a.zpw + ch);
#pragma unroll
                for (int jj = 0; jj < FP; ++jj) {
                    const int m = min(mbase + jj * 16, a.M - 1);
                    const int s3 = a.asum[m];
                    acc[i][jj] -= zw * v4i{s3, s3, s3, s3};
                }
            }
        }
#pragma unroll
        for (int i = 0; i < FC; ++i) {
            const int cl = wc * WTC + i * 16 + lchk * 4;   // channel inside the tile
            int mult[4], bconst[4], rndzp[4], shift[4];
            load_chan4(a.chan_in_lds, chan_lds, a.chan, c0 + cl, mult, bconst, rndzp, shift);
#pragma unroll
            for (int jj = 0; jj < FP; ++jj) {
                uint32_t packed;
                if (a.fast_rq) {
                    uint32_t u[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int v = (int)((uint32_t)acc[i][jj][e] + (uint32_t)bconst[e]);
                        const int t = (__mulhi(v, mult[e]) + rndzp[e]) >> (shift[e] & 31);   // shift - 32 for shift in [33, 53]
                        u[e] = (uint32_t)clamp_i32(t, a.lo_off, a.hi_off);
                    }
                    packed = (u[0] | (u[1] << 8) | (u[2] << 16) | (u[3] << 24)) ^ a.out_xor;
                } else {
                    packed = 0;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int v = (int)((uint32_t)acc[i][jj][e] + (uint32_t)bconst[e]);
                        const int o =
                            clamp_i(rounding_mul_shift(v, mult[e], shift[e], a.rounding) + a.zp_y, a.lo, a.hi);
                        packed |= ((uint32_t)o & 0xffu) << (8 * e);
                    }
                }
                const int pl = wpos * WTP + jj * 16 + lrow;      // pixel inside the tile
                *(uint32_t *)(stage + pl * SP + cl) = packed;
                acc[i][jj] = v4i{0, 0, 0, 0};
            }
        }
        __syncthreads();
        constexpr int CH = TC / 16;   // 16-byte chunks per pixel row
        const int kmax = a.K - c0;    // valid channels of this tile
#pragma unroll
        for (int it = 0; it < (TP * CH + NT - 1) / NT; ++it) {
            const int idx = it * NT + tid;
            if (idx < TP * CH) {
                const int pl = idx / CH, qc = idx % CH;
                const int m = p0 + pl;
                if (m < a.M && qc * 16 < kmax) {
                    const v4i v = *(const v4i *)(stage + pl * SP + qc * 16);
                    uint8_t *dst = (uint8_t *)a.y + (size_t)m * a.y_ldc + a.y_coff + c0 + qc * 16;
                    if (qc * 16 + 16 <= kmax) {
                        __builtin_nontemporal_store(v, (v4i *)dst);
                    } else {
                        for (int e = 0; e < kmax - qc * 16; ++e) {
                            const int w = e < 4 ? v.x : e < 8 ? v.y : e < 12 ? v.z : v.w;
                            dst[e] = (uint8_t)((uint32_t)w >> (8 * (e & 3)));
                        }
                    }
                }
            }
        }
    };

    // ---- prologue: fill the ring ----------------------------------------
    // Every stage issues its loads unconditionally (stages past the end of
    // the work re-read valid addresses of the last tile and are never
    // used), so the number of loads in flight behind each ring slot is the
    // same on every path and the compiler's wait before an LDS store covers
    // only that slot.
    begin_tile(0);
#pragma unroll
    for (int d = 0; d < D; ++d) {
        load_stage(ra[d], rb[d]);
        next_stage();
    }
    store_stage(0, ra[0], rb[0]);
    __syncthreads();

    // ---- main loop: D stages per trip so ring slots are compile-time -----
    int c_tile = 0, c_k = 0;   // compute position
    for (int g0 = 0; g0 < G; g0 += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            const int g = g0 + d;
            // refill this slot (stage g is already in LDS) with stage g + D
            load_stage(ra[d], rb[d]);
            next_stage();
            if (g < G) {
                const int8_t *As = lds[d & 1];
                const int8_t *Bs = lds[d & 1] + TC * BK;
#pragma unroll
                for (int kk = 0; kk < BK / 64; ++kk) {
                    const int chunkid = kk * 4 + lchk;
                    v4i fa[FC], fb[FP];
#pragma unroll
                    for (int i = 0; i < FC; ++i) {
                        const int row = wc * WTC + i * 16 + lrow;
                        fa[i] = *(const v4i *)(As + row * BK + ((chunkid ^ swizzle<CPR>(row)) << 4));
                    }
#pragma unroll
                    for (int jj = 0; jj < FP; ++jj) {
                        const int row = wpos * WTP + jj * 16 + lrow;
                        fb[jj] = *(const v4i *)(Bs + row * BK + ((chunkid ^ swizzle<CPR>(row)) << 4));
                    }
#pragma unroll
                    for (int i = 0; i < FC; ++i)
#pragma unroll
                        for (int jj = 0; jj < FP; ++jj)
                            acc[i][jj] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[jj], acc[i][jj], 0, 0, 0);
                }
            }
            store_stage((d + 1) & 1, ra[(d + 1) % D], rb[(d + 1) % D]);
            if (g < G && ++c_k == nk) {
                if (a.staged) {
                    __syncthreads();   // every wave is done reading lds[d & 1]
                    epilogue_staged(c_tile, lds[d & 1]);
                } else {
                    epilogue(c_tile);
                }
                c_k = 0;
                ++c_tile;
            }
            __syncthreads();
        }
    }
}

// Channel padding for C % 4 != 0: copies x into [N][H][W][C4] with the
// extra channels holding zp_x.  Padded channels contribute (zp_x - zp_x) * w
// = 0 to every accumulator, so the conv over C4 channels (J' = R*S*C4, zero
// weights in the extra channels) is the same conv.
__global__ void __launch_bounds__(256) pad_channels_kernel(const uint8_t *x, uint8_t *xp, long long pixels,
                                                           int C, int C4, uint8_t zp)
{
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= pixels * C4)
        return;
    const long long p = i / C4;
    const int c = (int)(i - p * C4);
    xp[i] = c < C ? x[p * C + c] : zp;
}

// Term 3 of Eq. (3): asum[m] = sum over the receptive field of x~' (the
// legalised input, zp_x' at padded taps).  Only needed when some zp_w != 0.
__global__ void __launch_bounds__(256) window_sum_kernel(ConvArgs a, int32_t *out)
{
    const int m = blockIdx.x * blockDim.x + threadIdx.x;
    if (m >= a.M)
        return;
    const int ow = m % a.Wo, t = m / a.Wo, oh = t % a.Ho, n = t / a.Ho;
    const int flip = (int)(a.flip4 & 0xffu);
    const int pad = (int)(int8_t)(uint8_t)(a.padbuf[0] ^ flip);
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

// Plan preparation: pack w[K][R*S][C] into [Kpad][Jpad] with each tap's
// channels padded from C to C4 (zeros in the extra channels, the K-tail and
// the extra rows), and fold bias, term 2 and term 4 into chan[k].bconst.
// The other chan fields and zpw were uploaded by the host.  One workgroup
// per (padded) output channel.
__global__ void __launch_bounds__(256) prep_conv_kernel(const int8_t *w, const int32_t *bias, int K, int RS,
                                                        int C, int C4, int Jpad, int32_t zpx, int8_t *wp,
                                                        ChanRec *chan, const int32_t *zpw)
{
    const int k = blockIdx.x;
    __shared__ long long part[256];
    long long sum = 0;
    for (int j = threadIdx.x; j < Jpad; j += blockDim.x) {
        const int tap = j / C4, c = j - tap * C4;
        int8_t v = 0;
        if (k < K && tap < RS && c < C)
            v = w[((size_t)k * RS + tap) * C + c];
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
    if (threadIdx.x == 0 && k < K) {
        const long long wsum = part[0];
        const long long b = bias ? (long long)bias[k] : 0;
        const long long J = (long long)RS * C4;
        const long long c = b - (long long)zpx * wsum + J * zpx * (long long)zpw[k];
        chan[k].bconst = (int32_t)(uint32_t)(unsigned long long)c;
    }
}

// Depth of the register prefetch ring (stages in flight): 4 where the
// staging registers fit beside the accumulators, 2 for the largest tiles.
template <int TC, int TP>
constexpr int ring_depth()
{
    return TC * TP >= 128 * 128 ? 2 : 4;
}

template <int TC, int TP, int BK, int WC, int WP, int AVEC>
static hipError_t launch_cfg(const ConvArgs &a, hipStream_t st)
{
    dim3 grid(a.nblocks), block(256);
    const unsigned dyn = a.chan_in_lds ? (unsigned)(a.Kpad * sizeof(ChanRec)) : 0u;
    launch_main((conv_mfma_kernel<TC, TP, BK, WC, WP, AVEC, ring_depth<TC, TP>()>), grid, block, dyn, st, a);
    return hipGetLastError();
}

template <int TC, int TP, int BK, int WC, int WP, int AVEC>
static int occupancy_cfg(size_t dyn)
{
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &n, conv_mfma_kernel<TC, TP, BK, WC, WP, AVEC, ring_depth<TC, TP>()>, 256, dyn) != hipSuccess)
        return 1;
    return n > 0 ? n : 1;
}

template <int TC, int TP, int BK, int WC, int WP>
static int occupancy_avec(int avec, size_t dyn)
{
    if (avec == 16) return occupancy_cfg<TC, TP, BK, WC, WP, 16>(dyn);
    if (avec == 8) return occupancy_cfg<TC, TP, BK, WC, WP, 8>(dyn);
    return occupancy_cfg<TC, TP, BK, WC, WP, 4>(dyn);
}

int conv_blocks_per_cu(int tile, int avec, size_t dyn)
{
    switch (tile) {
    case TILE_128x128: return occupancy_avec<128, 128, 128, 2, 2>(avec, dyn);
    case TILE_64x256: return occupancy_avec<64, 256, 128, 1, 4>(avec, dyn);
    case TILE_256x128: return occupancy_avec<256, 128, 128, 2, 2>(avec, dyn);
    case TILE_64x64: return occupancy_avec<64, 64, 128, 2, 2>(avec, dyn);
    case TILE_64x64_K64: return occupancy_avec<64, 64, 64, 2, 2>(avec, dyn);
    case TILE_128x128_K64: return occupancy_avec<128, 128, 64, 2, 2>(avec, dyn);
    case TILE_128x64: return occupancy_avec<128, 64, 128, 2, 2>(avec, dyn);
    case TILE_256x64_K64: return occupancy_avec<256, 64, 64, 4, 1>(avec, dyn);
    default: return occupancy_avec<64, 128, 128, 2, 2>(avec, dyn);
    }
}

template <int TC, int TP, int BK, int WC, int WP>
static hipError_t launch_avec(const ConvArgs &a, int avec, hipStream_t st)
{
    if (avec == 16) return launch_cfg<TC, TP, BK, WC, WP, 16>(a, st);
    if (avec == 8) return launch_cfg<TC, TP, BK, WC, WP, 8>(a, st);
    return launch_cfg<TC, TP, BK, WC, WP, 4>(a, st);
}

hipError_t launch_conv(const ConvArgs &a, int tile, int avec, hipStream_t st)
{
    switch (tile) {
    case TILE_128x128: return launch_avec<128, 128, 128, 2, 2>(a, avec, st);
    case TILE_64x256: return launch_avec<64, 256, 128, 1, 4>(a, avec, st);
    case TILE_256x128: return launch_avec<256, 128, 128, 2, 2>(a, avec, st);
    case TILE_64x64: return launch_avec<64, 64, 128, 2, 2>(a, avec, st);
    case TILE_64x64_K64: return launch_avec<64, 64, 64, 2, 2>(a, avec, st);
    case TILE_128x128_K64: return launch_avec<128, 128, 64, 2, 2>(a, avec, st);
    case TILE_128x64: return launch_avec<128, 64, 128, 2, 2>(a, avec, st);
    case TILE_256x64_K64: return launch_avec<256, 64, 64, 4, 1>(a, avec, st);
    default: return launch_avec<64, 128, 128, 2, 2>(a, avec, st);
    }
}

hipError_t launch_pad_channels(const uint8_t *x, uint8_t *xp, long long pixels, int C, int C4, uint8_t zp,
                               hipStream_t st)
{
    const long long n = pixels * C4;
    hipLaunchKernelGGL(pad_channels_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, x, xp, pixels, C,
                       C4, zp);
    return hipGetLastError();
}

hipError_t launch_window_sums(const ConvArgs &a, int32_t *out, hipStream_t st)
{
    dim3 grid((a.M + 255) / 256), block(256);
    hipLaunchKernelGGL(window_sum_kernel, grid, block, 0, st, a, out);
    return hipGetLastError();
}

hipError_t launch_prep_conv(const int8_t *w, const int32_t *bias, int K, int RS, int C, int C4, int Jpad,
                            int Kpad, int32_t zpx, int8_t *wp, ChanRec *chan, const int32_t *zpw, hipStream_t st)
{
    hipLaunchKernelGGL(prep_conv_kernel, dim3(Kpad), dim3(256), 0, st, w, bias, K, RS, C, C4, Jpad, zpx, wp,
                       chan, zpw);
    return hipGetLastError();
}

}  // namespace qnn
