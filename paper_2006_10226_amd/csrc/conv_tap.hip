// Implicit-GEMM quantized conv2d / dense for channel counts that are a
// multiple of the K-step (64 or 128 bytes): the fast path of the conv.
//
// Same arithmetic as conv_mfma.hip (Jain et al., Sec. II-B Eq. (3), Sec.
// III-B/C: term 1 on int8 MFMA over the legalised input x' = x - 128, terms
// 2 and 4 and the bias folded into ChanRec.bconst, term 3 from the window
// sums, requantize of Eq. (5) in the epilogue); what differs is how the
// operands reach the matrix cores.  Because C % BK == 0, every K-step reads
// a single filter tap (r, s) and a channel range [cc, cc + BK) of it, so
// the address of every gathered 16-byte chunk is
//     x + pixel_base(m) + tap_offset(r, s) + cc + 16 * q
// with pixel_base per thread and tile, tap_offset uniform, and cc uniform.
// The loads are raw buffer loads: the per-thread part is the VGPR offset,
// cc the scalar offset.  A tap outside the image gets an offset past the
// end of the buffer, which the hardware answers with zero bytes without
// touching memory; XOR-ing those zeros with zp_x' instead of with the
// uint8 -> int8 flip gives exactly the zero-point padding of Sec. III-B.
// Per K-step the loader therefore spends a few instructions per tap change
// and one XOR per gathered dword, instead of recomputing coordinates.
//
// Tiles are large (TC x TP = 128 x 128 and up, 64 x 64 per wave), because a
// CU streams roughly 64 bytes per clock from L1/L2 while its matrix cores
// consume 8192 int8 ops per clock: a tile must perform over 128 ops per
// byte loaded to keep them busy.  Two register stages of prefetch and two
// LDS stages overlap the loads with the MFMAs, one barrier per K-step.
#include "conv_common.h"

namespace qnn {

using namespace conv;

__device__ __forceinline__ v4i bload(__amdgpu_buffer_rsrc_t r, int voff, int soff)
{
    return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
}

// Occupancy the register budget is sized for: wave tiles of 128 x 64 need
// all 512 registers of a SIMD lane (accumulators in AGPRs), smaller ones
// leave room for a second workgroup.
template <int WTC, int WTP>
constexpr int tap_occupancy()
{
    return WTC * WTP >= 128 * 64 ? 1 : 2;
}

// FUSE: the epilogue applies the residual add (store_tile).
template <int TC, int TP, int BK, int WC, int WP, bool FUSE = false>
__global__ void __launch_bounds__(WC *WP * 64, (tap_occupancy<TC / WC, TP / WP>())) conv_tap_kernel(ConvArgs a)
{
    constexpr int NT = WC * WP * 64;
    constexpr int CPR = BK / 16;                // 16-byte chunks per LDS row
    constexpr int RPP = NT / CPR;               // rows per load pass of the workgroup
    constexpr int A_PASS = TC / RPP;            // weight rows per thread
    constexpr int B_PASS = TP / RPP;            // pixel rows per thread
    constexpr int WTC = TC / WC, WTP = TP / WP; // wave tile
    constexpr int FC = WTC / 16, FP = WTP / 16; // 16x16 blocks per wave
    constexpr int STAGE = (TC + TP) * BK;
    static_assert(BK == 64 || BK == 128, "K-step");
    static_assert(TC % RPP == 0 && TP % RPP == 0, "tile rows must fill the load passes");
    static_assert(WTC % 16 == 0 && WTP % 16 == 0, "wave tile");

    __shared__ __attribute__((aligned(16))) int8_t lds[2 * STAGE];
    // the tile's channel records, fetched at the start for the epilogue
    __shared__ __attribute__((aligned(16))) ChanRec recs[TC];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave
    const int wc = wave / WP, wpos = wave % WP;

    // Workgroups are dealt round-robin to the 8 XCDs; XCD x takes the x-th
    // eighth of the tile list, so the channel tiles of one pixel tile (which
    // share its activations) meet in one L2.
    const int chunk = (a.ntiles + 7) >> 3;
    const int xcd = blockIdx.x & 7;
    const int tile = xcd * chunk + (blockIdx.x >> 3);
    if (tile >= min(a.ntiles, (xcd + 1) * chunk))
        return;
    const int c0 = (tile % a.tiles_c) * TC;
    const int p0 = (tile / a.tiles_c) * TP;

    const int q = tid % CPR;        // 16-byte chunk this thread loads
    const int rbase = tid / CPR;    // first tile row this thread loads

    const __amdgpu_buffer_rsrc_t rx =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.x, (short)0, a.N * a.H * a.W * a.C, kBufFlags);
    const __amdgpu_buffer_rsrc_t rw =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.wp, (short)0, a.Kpad * a.Jpad, kBufFlags);
    if (wave == WC * WP - 1) {
        // records c0 .. c0 + TC - 1 (c0 + TC <= Kpad), a kilobyte per load
        const __amdgpu_buffer_rsrc_t rc =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.chan, (short)0, a.Kpad * (int)sizeof(ChanRec), kBufFlags);
#pragma unroll
        for (int q = 0; q < TC / 64; ++q)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rc, (__attribute__((address_space(3))) void *)(recs + q * 64), 16,
                                                     (c0 + q * 64 + lane) * (int)sizeof(ChanRec), 0, 0, 0);
    }

    int voffA[A_PASS];
#pragma unroll
    for (int i = 0; i < A_PASS; ++i)
        voffA[i] = (c0 + rbase + i * RPP) * a.Jpad + q * 16;

    // per pixel row: byte offset of tap (0, 0) (negative inside the top or
    // left padding) and the taps that fall inside the image: bit r of the
    // low half for rows, bit s of the high half for columns
    int pbase[B_PASS];
    uint32_t pmask[B_PASS];
#pragma unroll
    for (int i = 0; i < B_PASS; ++i) {
        const int m = p0 + rbase + i * RPP;
        pbase[i] = 0;
        pmask[i] = 0;
        if (m < a.M) {
            const int ow = m % a.Wo, t = m / a.Wo;
            const int oh = t % a.Ho, n = t / a.Ho;
            const int ih0 = oh * a.sh - a.pt, iw0 = ow * a.sw - a.pl;
            pbase[i] = ((n * a.H + ih0) * a.W + iw0) * a.C + q * 16;
            uint32_t rm = 0, cm = 0;
            for (int r = 0; r < a.R; ++r)
                rm |= (uint32_t)((unsigned)(ih0 + r * a.dh) < (unsigned)a.H) << r;
            for (int s = 0; s < a.S; ++s)
                cm |= (uint32_t)((unsigned)(iw0 + s * a.dw) < (unsigned)a.W) << s;
            pmask[i] = rm | (cm << 16);
        }
    }

    // ---- loader: tap (lr, ls), channel offset lc of the next stage ------
    const int nk = a.nk;
    const uint32_t flip4 = a.flip4, zp4 = a.zp4;
    int lr = 0, ls = 0, lc = 0;
    int voffB[B_PASS];
    uint32_t xmask[B_PASS];
    auto set_tap = [&]() {
        const int toff = (lr * a.dh * a.W + ls * a.dw) * a.C;
        const uint32_t rin = lr < a.R ? 1u : 0u;
#pragma unroll
        for (int i = 0; i < B_PASS; ++i) {
            const bool v = (pmask[i] >> lr) & (pmask[i] >> (16 + ls)) & rin;
            voffB[i] = v ? pbase[i] + toff : kOutOfRange;
            xmask[i] = v ? flip4 : zp4;
        }
    };
    // Loads are issued unconditionally, also for the two stages past the
    // end: those read out of range (zeros, no memory traffic) and are never
    // used, and the uniform load count keeps the compiler's waits exact.
    // Out of range is always signalled in the VGPR offset (>= 2^31, beyond
    // any buffer here) with a small scalar offset, so the hardware's range
    // check sees it whether or not it includes the scalar offset.
    auto load = [&](v4i (&A)[A_PASS], v4i (&B)[B_PASS], uint32_t (&X)[B_PASS], int ks) {
        // (the scalar offsets are uniform; readfirstlane tells the compiler)
        const bool live = ks < nk;
        const int soffA = __builtin_amdgcn_readfirstlane(live ? ks * BK : 0);
        const int oobA = __builtin_amdgcn_readfirstlane(live ? 0 : kOutOfRange);
        const int soffB = __builtin_amdgcn_readfirstlane(lc);
#pragma unroll
        for (int i = 0; i < A_PASS; ++i)
            A[i] = bload(rw, voffA[i] | oobA, soffA);
#pragma unroll
        for (int i = 0; i < B_PASS; ++i) {
            B[i] = bload(rx, voffB[i], soffB);
            X[i] = xmask[i];
        }
        lc += BK;
        if (lc == a.C) {
            lc = 0;
            if (++ls == a.S) {
                ls = 0;
                ++lr;   // lr == R past the last tap: every row reads out of range
            }
            set_tap();
        }
    };
    auto store = [&](int buf, const v4i (&A)[A_PASS], const v4i (&B)[B_PASS], const uint32_t (&X)[B_PASS]) {
        int8_t *As = lds + buf * STAGE;
        int8_t *Bs = As + TC * BK;
#pragma unroll
        for (int i = 0; i < A_PASS; ++i) {
            const int row = rbase + i * RPP;
            *(v4i *)(As + row * BK + ((q ^ swz<CPR>(row)) << 4)) = A[i];
        }
#pragma unroll
        for (int i = 0; i < B_PASS; ++i) {
            const int row = rbase + i * RPP;
            const int xm = (int)X[i];
            *(v4i *)(Bs + row * BK + ((q ^ swz<CPR>(row)) << 4)) = B[i] ^ v4i{xm, xm, xm, xm};
        }
    };

    // ---- MFMAs over one LDS stage --------------------------------------
    const int lrow = lane & 15;   // operand row inside a 16-row block
    const int lchk = lane >> 4;   // 16-byte chunk inside a 64-byte k slice
    const int lsw = swz<CPR>(lrow);
    v4i acc[FC][FP];
#pragma unroll
    for (int i = 0; i < FC; ++i)
#pragma unroll
        for (int j = 0; j < FP; ++j)
            acc[i][j] = v4i{0, 0, 0, 0};
    auto compute = [&](int buf) {
        const int8_t *As = lds + buf * STAGE + (wc * WTC + lrow) * BK;
        const int8_t *Bs = lds + buf * STAGE + TC * BK + (wpos * WTP + lrow) * BK;
#pragma unroll
        for (int kk = 0; kk < BK / 64; ++kk) {
            const int co = ((kk * 4 + lchk) ^ lsw) << 4;
            v4i fa[FC], fb[FP];
#pragma unroll
            for (int i = 0; i < FC; ++i)
                fa[i] = *(const v4i *)(As + i * 16 * BK + co);
#pragma unroll
            for (int j = 0; j < FP; ++j)
                fb[j] = *(const v4i *)(Bs + j * 16 * BK + co);
#pragma unroll
            for (int i = 0; i < FC; ++i)
#pragma unroll
                for (int j = 0; j < FP; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
        }
    };

    // ---- pipeline: stage k in LDS, k + 1 and k + 2 in registers ----------
    // Two K-steps per trip so the register stages have fixed names; a trip
    // starts with stage k in LDS buffer 0 and stage k + 1 loading into R*1.
    v4i RA0[A_PASS], RB0[B_PASS], RA1[A_PASS], RB1[B_PASS];
    uint32_t X0[B_PASS], X1[B_PASS];
    set_tap();
    load(RA0, RB0, X0, 0);
    load(RA1, RB1, X1, 1);
    store(0, RA0, RB0, X0);
    // the record loads are older than stage 0's, whose data store() waited
    // for; the barrier publishes them
    __syncthreads();
    add_bconst<TC, TP, WC, WP>(acc, recs);
    int k = 0;
    for (; k + 2 <= nk; k += 2) {
        load(RA0, RB0, X0, k + 2);
        compute(0);                   // stage k
        store(1, RA1, RB1, X1);       // stage k + 1
        __syncthreads();
        load(RA1, RB1, X1, k + 3);
        compute(1);                   // stage k + 1
        store(0, RA0, RB0, X0);       // stage k + 2
        __syncthreads();
    }
    if (k < nk) {                     // odd step count: the last stage is in buffer 0
        compute(0);
        __syncthreads();
    }

    // the record loads (LDS-direct) have landed before anyone reads them
    __builtin_amdgcn_s_waitcnt((0) | (7 << 4) | (15 << 8) | (0 << 14));
    __syncthreads();
    store_tile<TC, TP, WC, WP, 2 * STAGE, FUSE>(a, acc, lds, c0, p0, recs);
}

// TapTile -> tile, K-step and wave grid.
struct TapCfg {
    int tc, tp, bk, wc, wp;
};
static constexpr TapCfg kTapCfg[TAP_COUNT] = {
    {128, 128, 64, 2, 2},  {256, 128, 64, 4, 2},  {128, 256, 64, 2, 4},  {128, 128, 128, 2, 2},
    {256, 128, 128, 4, 2}, {128, 256, 128, 2, 4}, {64, 128, 128, 1, 4},  {128, 64, 128, 4, 1},
    {256, 128, 128, 2, 2}, {128, 256, 128, 2, 2}, {256, 128, 64, 2, 2},  {128, 256, 64, 2, 2},
};

TileShape tap_tile_shape(int tile)
{
    const TapCfg &c = kTapCfg[tile];
    return {c.tc, c.tp, c.bk};
}

int tap_wave_tile(int tile)
{
    return kTapCfg[tile].tc / kTapCfg[tile].wc * (kTapCfg[tile].tp / kTapCfg[tile].wp);
}

int tap_threads(int tile)
{
    return kTapCfg[tile].wc * kTapCfg[tile].wp * 64;
}

template <int T>
static hipError_t launch_tap_cfg(const ConvArgs &a, hipStream_t st)
{
    constexpr TapCfg c = kTapCfg[T];
    const int grid = (a.ntiles + 7) / 8 * 8;
    if (a.res) {
        if constexpr (c.tc / c.wc * (c.tp / c.wp) <= kFuseMaxWaveTile)
            launch_main((conv_tap_kernel<c.tc, c.tp, c.bk, c.wc, c.wp, true>), dim3(grid), dim3(c.wc * c.wp * 64),
                        0, st, a);
        else
            return hipErrorInvalidValue;   // no fused-add instantiation
    } else {
        launch_main((conv_tap_kernel<c.tc, c.tp, c.bk, c.wc, c.wp>), dim3(grid), dim3(c.wc * c.wp * 64), 0, st,
                    a);
    }
    return hipGetLastError();
}

template <int T>
static hipError_t launch_tap_from(const ConvArgs &a, int tile, hipStream_t st)
{
    if constexpr (T < TAP_COUNT) {
        if (tile == T)
            return launch_tap_cfg<T>(a, st);
        return launch_tap_from<T + 1>(a, tile, st);
    } else {
        return hipErrorInvalidValue;
    }
}

hipError_t launch_conv_tap(const ConvArgs &a, int tile, hipStream_t st)
{
    return launch_tap_from<0>(a, tile, st);
}

}  // namespace qnn
