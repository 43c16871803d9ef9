// Persistent streaming variant of the LDS-direct conv kernel (conv_dma.hip)
// for channel counts that are a multiple of 64.
//
// Arithmetic as in conv_dma.hip (Jain et al., Sec. II-B Eq. (3), Sec.
// III-B/C): term 1 on int8 MFMA, terms 2 and 4 and the bias in
// ChanRec.bconst, term 3 from the window sums, the padding correction of
// the zero-filled gathers per border class, requantize of Eq. (5) fused in
// the epilogue.
//
// What differs is the schedule.  A workgroup stays resident and walks a
// list of output tiles of one channel tile, and a single stage ring runs
// through the K-steps of all of them, so the loads of the next tile are in
// flight while the current one finishes its MFMAs, requantizes and stores.
// Layers with short reductions (1x1 convolutions with few input channels,
// one to eight K-steps per tile) are bound by memory latency in the
// one-tile-per-workgroup kernel; here the memory pipe never drains between
// tiles.
//
// Waves are specialised: NL loader waves issue every LDS-direct load and
// nothing else, NW compute waves read fragments, run the MFMAs and issue
// every store.  The vector-memory counter of a loader wave therefore counts
// loads only and can be waited on at any depth; the stores of the compute
// waves are never waited for.  All waves meet at one barrier per K-step and
// one more per tile (between the staging writes and reads of the
// epilogue).
#include "conv_common.h"

namespace qnn {

using namespace conv;

namespace {

template <int N>
__device__ __forceinline__ void wait_vm()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// lgkmcnt(0): this wave's LDS reads have returned and its LDS writes are done.
__device__ __forceinline__ void wait_lgkm0()
{
    __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
}

__device__ __forceinline__ void barrier()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Swizzle of 64-byte LDS rows, as in conv_dma.hip (measured conflict free).
__device__ __forceinline__ int sw64(int row)
{
    return (row >> 1) & 3;
}

__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, int8_t *lds_dst, int voff, int soff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void *)lds_dst, 16, voff, soff, 0,
                                             0);
}

// Bit t (t < n <= 16) set when 0 <= i0 + t * d < L: the filter rows (or
// columns) of a window that fall inside the image.  Undilated filters (d
// uniformly 1) take the closed form, others a loop.
__device__ __forceinline__ uint32_t inside_bits(int i0, int d, int n, int L)
{
    if (d == 1) {
        const int lo = max(0, -i0), hi = min(n - 1, L - 1 - i0);
        return hi < lo ? 0u : ((2u << hi) - 1u) & ~((1u << lo) - 1u);
    }
    uint32_t m = 0;
    for (int t = 0; t < n; ++t)
        m |= (uint32_t)((unsigned)(i0 + t * d) < (unsigned)L) << t;
    return m;
}

}  // namespace

// Tiles of workgroup b: XCD x = b % 8 owns tiles [x * chunk, (x + 1) * chunk)
// and its nx = grid / 8 workgroups deal them out in turn, so at any moment
// the workgroups of one XCD work on nx consecutive tiles, i.e. on all
// channel tiles of a few pixel tiles, and share the activations in their
// L2.  nx is a multiple of tiles_c, hence every tile of a workgroup has the
// same channel tile.
template <int TC, int TP, int WC, int WP, int NL, int NS, bool FLIP>
__global__ void __launch_bounds__((WC * WP + NL) * 64, 3) conv_stream_kernel(ConvArgs a)
{
    constexpr int NW = WC * WP;           // compute waves
    constexpr int NTC = NW * 64;          // compute threads
    constexpr int BK = 64;
    constexpr int WTC = TC / WC, WTP = TP / WP;
    constexpr int FC = WTC / 16, FP = WTP / 16;
    constexpr int STAGE = (TC + TP) * BK;
    constexpr int LA = TC / (16 * NL);    // 1 KB weight blocks per loader wave per stage
    constexpr int LB = TP / (16 * NL);    // 1 KB activation blocks per loader wave per stage
    constexpr int LPS = LA + LB;          // loads per loader lane per stage
    constexpr int SP = TC + 16;           // staging row pitch (bytes)
    constexpr int RING = NS * STAGE;
    constexpr int STG = TP * SP;
    static_assert(TC % (16 * NL) == 0 && TP % (16 * NL) == 0, "loader waves fetch whole 16-row blocks");
    static_assert(NS >= 3, "two stages in flight beyond the one being read");
    static_assert(LPS * (NS - 1) < 64, "vmcnt range");

    __shared__ __attribute__((aligned(1024))) int8_t lds[RING + STG + TC * 16 + TC * 4];
    extern __shared__ __attribute__((aligned(16))) int32_t pcorr_lds[];   // [ncls + 1][TC] when a.pcorr
    int8_t *const stg = lds + RING;
    const ChanRec *const chn = (const ChanRec *)(lds + RING + STG);
    int32_t *const zwl = (int32_t *)(lds + RING + STG + TC * 16);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave

    const int nx = gridDim.x >> 3;
    const int xcd = blockIdx.x & 7;
    const int tbeg = xcd * a.chunk + (blockIdx.x >> 3);
    const int tend = min(a.ntiles, (xcd + 1) * a.chunk);
    const int ntl = tbeg < tend ? (tend - tbeg + nx - 1) / nx : 0;
    if (ntl == 0)
        return;
    const int c0 = (tbeg % a.tiles_c) * TC;
    // pixel tile of the workgroup's i-th tile: pt0 + i * pstep
    const int pt0 = tbeg / a.tiles_c, pstep = nx / a.tiles_c;
    const int nk = a.nk;
    const int G = ntl * nk;   // K-steps of this workgroup over all its tiles

    if (wave >= NW) {
        // ================================================================ loader
        const int lw = wave - NW;
        const __amdgpu_buffer_rsrc_t rx =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.x, (short)0, a.N * a.H * a.W * a.C, kBufFlags);
        const __amdgpu_buffer_rsrc_t rw =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.wp, (short)0, a.Kpad * a.Jpad, kBufFlags);
        // lane L of a 16-row block writes LDS byte 16 * L: row L / 4,
        // physical chunk L % 4, holding logical chunk (L % 4) ^ sw64(row)
        const int r16 = lane >> 2, pch = lane & 3;
        int voffA[LA];
#pragma unroll
        for (int i = 0; i < LA; ++i) {
            const int row = (i * NL + lw) * 16 + r16;
            voffA[i] = (c0 + row) * a.Jpad + ((pch ^ sw64(row)) << 4);
        }
        int pbase[LB], voffB[LB];
        uint32_t pmask[LB];
        int li = 0, lk = 0, lr = 0, ls = 0, lc = 0;
        auto set_tap = [&]() __attribute__((always_inline)) {
            const int toff = a.rowpack ? lr * 2 * a.row_bytes : (lr * a.dh * a.W + ls * a.dw) * a.C;
            const uint32_t rin = lr < a.R ? 1u : 0u;
#pragma unroll
            for (int i = 0; i < LB; ++i) {
                const bool v = (pmask[i] >> lr) & (pmask[i] >> (16 + ls)) & rin;
                voffB[i] = v ? pbase[i] + toff : kOutOfRange;
            }
        };
        // pixel rows of tile li of this workgroup (none past the last tile)
        auto setup_tile = [&]() __attribute__((always_inline)) {
            const int p0 = (pt0 + li * pstep) * TP;
            const bool live = li < ntl;
#pragma unroll
            for (int i = 0; i < LB; ++i) {
                const int row = (i * NL + lw) * 16 + r16;
                const int m = p0 + row;
                pbase[i] = 0;
                pmask[i] = 0;
                if (live && m < a.M) {
                    const int t = fast_div(m, a.mWo, a.sWo);
                    const int ow = m - t * a.Wo;
                    const int n = fast_div(t, a.mHo, a.sHo);
                    const int oh = t - n * a.Ho;
                    const int q = pch ^ sw64(row);
                    if (a.rowpack) {
                        // K-step s: filter rows 2s, 2s + 1 of the padded image,
                        // logical chunk q = row q / 2, half q % 2
                        pbase[i] = ((n * a.H + oh * a.sh) * a.W + ow * a.sw) * a.C + (q >> 1) * a.row_bytes +
                                   (q & 1) * 16;
                        pmask[i] = 0xffffffffu;
                    } else {
                        const int ih0 = oh * a.sh - a.pt, iw0 = ow * a.sw - a.pl;
                        pbase[i] = ((n * a.H + ih0) * a.W + iw0) * a.C + (q << 4);
                        pmask[i] = inside_bits(ih0, a.dh, a.R, a.H) | (inside_bits(iw0, a.dw, a.S, a.W) << 16);
                    }
                }
            }
            lr = 0;
            ls = 0;
            lc = 0;
            set_tap();
        };
        // Stages past the last tile are issued too, out of range (zeros, no
        // memory traffic), so every step waits for the same count.
        int lbuf = 0;
        auto issue = [&]() __attribute__((always_inline)) {
            int8_t *base = lds + lbuf * STAGE;
            lbuf = lbuf + 1 == NS ? 0 : lbuf + 1;
            const bool live = li < ntl;
            const int soffA = __builtin_amdgcn_readfirstlane(live ? lk * BK : 0);
            const int oobA = __builtin_amdgcn_readfirstlane(live ? 0 : kOutOfRange);
            const int soffB = __builtin_amdgcn_readfirstlane(lc);
#pragma unroll
            for (int i = 0; i < LA; ++i)
                dma16(rw, base + (i * NL + lw) * 16 * BK, voffA[i] | oobA, soffA);
#pragma unroll
            for (int i = 0; i < LB; ++i)
                dma16(rx, base + TC * BK + (i * NL + lw) * 16 * BK, voffB[i], soffB);
            if (++lk == nk) {
                lk = 0;
                ++li;
                setup_tile();
            } else if (a.rowpack) {
                ++lr;
                set_tap();
            } else {
                lc += BK;
                if (lc == a.C) {
                    lc = 0;
                    if (++ls == a.S) {
                        ls = 0;
                        ++lr;
                    }
                    set_tap();
                }
            }
        };

        setup_tile();
#pragma unroll 1
        for (int s = 0; s < NS; ++s)
            issue();
        wait_vm<LPS *(NS - 1)>();   // stage 0 has landed
        barrier();
        int kk = 0;
        for (int g = 0; g < G; ++g) {
            // barrier of step g: stage g + 1 has landed, every compute wave
            // is done reading stage g, whose buffer takes stage g + NS
            wait_vm<LPS *(NS - 2)>();
            barrier();
            issue();
            if (++kk == nk) {
                kk = 0;
                barrier();   // the epilogue's staging barrier
            }
        }
        wait_vm<0>();   // the last loads also write LDS
        return;
    }

    // ==================================================================== compute
    const int wc = wave / WP, wpos = wave % WP;
    const int lrow = lane & 15, lchk = lane >> 4;
    const int co = (lchk ^ sw64(lrow)) << 4;

    // per-channel tables of this workgroup's channel tile into LDS: the
    // requantize record with the shift stored as shift - 32 (the 32-bit
    // requantize path is the only one of this kernel), the weight zero
    // points, and the border-class correction rows plus a zero row for
    // interior pixels
    for (int i = tid; i < TC; i += NTC) {
        v4i r = *(const v4i *)(a.chan + c0 + i);
        r.w -= 32;
        ((v4i *)chn)[i] = r;
    }
    if (a.asum)
        for (int i = tid; i < TC; i += NTC)
            zwl[i] = a.zpw[c0 + i];
    if (a.pcorr)
        for (int i = tid; i < (a.ncls + 1) * TC; i += NTC) {
            const int cls = i / TC;
            pcorr_lds[i] = cls < a.ncls ? a.pcorr[(size_t)cls * a.Kpad + c0 + (i - cls * TC)] : 0;
        }

    // per-pixel data of the epilogue (border class row, window sum),
    // fetched one tile ahead
    int pxc[FP], pxs[FP];
    auto load_px = [&](int p0) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < FP; ++j) {
            const int m = p0 + wpos * WTP + j * 16 + lrow;
            if (a.pcorr) {
                const int c = m < a.M ? (int)a.pcls[m] : 255;
                pxc[j] = c == 255 ? a.ncls : c;
            }
            if (a.asum)
                pxs[j] = a.asum[min(m, a.M - 1)];
        }
    };
    int ti = 0;
    int p0 = pt0 * TP;
    load_px(p0);

    // accumulators start at the folded constant of their channel
    wait_lgkm0();
    barrier();   // stage 0 has landed; tables are in LDS
    v4i acc[FC][FP];
#pragma unroll
    for (int i = 0; i < FC; ++i) {
        const int cl = wc * WTC + i * 16 + lchk * 4;
        const v4i b = v4i{((const v4i *)chn)[cl].y, ((const v4i *)chn)[cl + 1].y, ((const v4i *)chn)[cl + 2].y,
                          ((const v4i *)chn)[cl + 3].y};
#pragma unroll
        for (int j = 0; j < FP; ++j)
            acc[i][j] = b;
    }
    v4i fa[2][FC], fb[2][FP];
    int rbuf = 0;
    auto read_frags = [&](v4i (&A)[FC], v4i (&B)[FP]) __attribute__((always_inline)) {
        const int8_t *As = lds + rbuf * STAGE + (wc * WTC + lrow) * BK + co;
        const int8_t *Bs = lds + rbuf * STAGE + TC * BK + (wpos * WTP + lrow) * BK + co;
        rbuf = rbuf + 1 == NS ? 0 : rbuf + 1;
#pragma unroll
        for (int i = 0; i < FC; ++i)
            A[i] = *(const v4i *)(As + i * 16 * BK);
#pragma unroll
        for (int j = 0; j < FP; ++j)
            B[j] = *(const v4i *)(Bs + j * 16 * BK);
    };
    auto mfma = [&](const v4i (&A)[FC], v4i (&B)[FP]) __attribute__((always_inline)) {
        if constexpr (FLIP) {
#pragma unroll
            for (int j = 0; j < FP; ++j)
                B[j] ^= v4i{(int)0x80808080, (int)0x80808080, (int)0x80808080, (int)0x80808080};
        }
#pragma unroll
        for (int i = 0; i < FC; ++i)
#pragma unroll
            for (int j = 0; j < FP; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A[i], B[j], acc[i][j], 0, 0, 0);
    };
    // Requantize the finished tile into the staging rows, meet the loader
    // at the staging barrier, store whole 16-byte row chunks.
    const int kmax = a.K - c0;
    auto epilogue = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < FC; ++i) {
            const int cl = wc * WTC + i * 16 + lchk * 4;
            v4i rec[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                rec[e] = ((const v4i *)chn)[cl + e];
            v4i zw = v4i{0, 0, 0, 0};
            if (a.asum)
                zw = *(const v4i *)(zwl + cl);
#pragma unroll
            for (int j = 0; j < FP; ++j) {
                v4i v = acc[i][j];
                if (a.pcorr)
                    v += *(const v4i *)(pcorr_lds + pxc[j] * TC + cl);
                if (a.asum)
                    v -= zw * v4i{pxs[j], pxs[j], pxs[j], pxs[j]};
                // 32-bit requantize (see requant4), bconst already in v
                uint32_t packed = 0;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int t = (__mulhi(v[e], rec[e].x) + rec[e].z) >> rec[e].w;
                    packed |= (uint32_t)min(max(t, a.lo_off), a.hi_off) << (8 * e);
                }
                const int pl = wpos * WTP + j * 16 + lrow;
                *(uint32_t *)(stg + pl * SP + cl) = packed ^ a.out_xor;
                acc[i][j] = v4i{rec[0].y, rec[1].y, rec[2].y, rec[3].y};
            }
        }
        wait_lgkm0();
        barrier();
        constexpr int CH = TC / 16;
#pragma unroll
        for (int it = 0; it < (TP * CH + NTC - 1) / NTC; ++it) {
            const int idx = it * NTC + tid;
            if (idx < TP * CH) {
                const int pl = idx / CH, qc = idx % CH;
                const int m = p0 + pl;
                if (m < a.M && qc * 16 < kmax) {
                    const v4i v = *(const v4i *)(stg + pl * SP + qc * 16);
                    uint8_t *dst = (uint8_t *)a.y + (size_t)m * a.y_ldc + a.y_coff + c0 + qc * 16;
                    if (a.staged && qc * 16 + 16 <= kmax) {   // 16-byte aligned rows
                        *(v4i *)dst = v;
                    } else {
                        for (int e = 0; e < 16 && qc * 16 + e < kmax; ++e)
                            dst[e] = (uint8_t)((uint32_t)v[e >> 2] >> (8 * (e & 3)));
                    }
                }
            }
        }
        ++ti;
        p0 += pstep * TP;
        if (ti < ntl)
            load_px(p0);
    };

    // One copy of the step (and of the epilogue) keeps the kernel small
    // enough for the instruction cache: the fragments of stage g + 1 are
    // read into the spare set while the MFMAs of stage g run, then moved.
    read_frags(fa[0], fb[0]);
    int kk = 0;
#pragma unroll 1
    for (int g = 0; g < G; ++g) {
        wait_lgkm0();
        barrier();
        read_frags(fa[1], fb[1]);
        mfma(fa[0], fb[0]);
        if (++kk == nk) {
            kk = 0;
            epilogue();
        }
#pragma unroll
        for (int i = 0; i < FC; ++i)
            fa[0][i] = fa[1][i];
#pragma unroll
        for (int j = 0; j < FP; ++j)
            fb[0][j] = fb[1][j];
    }
}

// StreamTile -> tile, compute wave grid, loader waves, stage count.
struct StreamCfg {
    int tc, tp, wc, wp, nl, ns;
};
static constexpr StreamCfg kStreamCfg[STREAM_COUNT] = {
    {64, 128, 2, 2, 2, 5},
    {64, 64, 2, 2, 1, 8},
    {128, 64, 2, 2, 1, 5},
    {128, 128, 2, 2, 2, 4},
};

TileShape stream_tile_shape(int tile)
{
    return {kStreamCfg[tile].tc, kStreamCfg[tile].tp, 64};
}

int stream_threads(int tile)
{
    return (kStreamCfg[tile].wc * kStreamCfg[tile].wp + kStreamCfg[tile].nl) * 64;
}

int stream_stages(int tile)
{
    return kStreamCfg[tile].ns;
}

template <int T>
static hipError_t launch_stream_cfg(const ConvArgs &a, hipStream_t st)
{
    constexpr StreamCfg c = kStreamCfg[T];
    const size_t dyn = a.pcorr ? (size_t)(a.ncls + 1) * c.tc * sizeof(int32_t) : 0;
    const dim3 block((c.wc * c.wp + c.nl) * 64);
    if (a.flip4)
        hipLaunchKernelGGL((conv_stream_kernel<c.tc, c.tp, c.wc, c.wp, c.nl, c.ns, true>), dim3(a.nblocks), block,
                           dyn, st, a);
    else
        hipLaunchKernelGGL((conv_stream_kernel<c.tc, c.tp, c.wc, c.wp, c.nl, c.ns, false>), dim3(a.nblocks), block,
                           dyn, st, a);
    return hipGetLastError();
}

template <int T>
static int stream_occupancy_cfg(size_t dyn)
{
    constexpr StreamCfg c = kStreamCfg[T];
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, conv_stream_kernel<c.tc, c.tp, c.wc, c.wp, c.nl, c.ns, true>,
                                                     stream_threads(T), dyn) != hipSuccess)
        return 0;
    return n > 0 ? n : 0;
}

template <int T>
static hipError_t launch_stream_from(const ConvArgs &a, int tile, hipStream_t st)
{
    if constexpr (T < STREAM_COUNT) {
        if (tile == T)
            return launch_stream_cfg<T>(a, st);
        return launch_stream_from<T + 1>(a, tile, st);
    } else {
        return hipErrorInvalidValue;
    }
}

template <int T>
static int stream_blocks_from(int tile, size_t dyn)
{
    if constexpr (T < STREAM_COUNT) {
        if (tile == T)
            return stream_occupancy_cfg<T>(dyn);
        return stream_blocks_from<T + 1>(tile, dyn);
    } else {
        return 0;
    }
}

hipError_t launch_conv_stream(const ConvArgs &a, int tile, hipStream_t st)
{
    if (tile < 0 || tile >= STREAM_COUNT || a.nblocks <= 0 || a.nblocks % 8 != 0 || a.mode != OUT_REQUANT ||
        !a.fast_rq)
        return hipErrorInvalidValue;
    return launch_stream_from<0>(a, tile, st);
}

int stream_blocks_per_cu(int tile, size_t dyn_lds)
{
    return stream_blocks_from<0>(tile, dyn_lds);
}

}  // namespace qnn
