// Implicit-GEMM quantized conv2d for stride-1, undilated 3x3 filters with
// C % 64 == 0, output rows of at most 64 pixels and more input channels
// than fit in LDS as resident weights (the deep ResNet stages).  A
// workgroup keeps the input window of NB output bands resident in LDS and
// streams its TC output channels' weights through LDS in groups of KS
// 64-channel slices, two groups in flight; wave (b, ks) accumulates band b
// over the slices ks, ks + KS, ... and the KS partial sums of a band are
// added through LDS before the epilogue.
//
// Arithmetic as in conv_mfma.hip (Jain et al., Sec. II-B Eq. (3), Sec.
// III-B/C): term 1 on int8 MFMA over x' (uint8 legalised by XOR 0x80),
// terms 2 and 4 and the bias in ChanRec.bconst (the accumulators of the
// ks = 0 waves start there), term 3 from the window sums, requantize of
// Eq. (5) in the epilogue.
//
// Bands.  A band is TR = min(Ho, 64 / Wo) whole output rows of one image
// (at most 64 pixels).  When an image has several bands, the NB bands of a
// workgroup are consecutive bands of one image and share one window of
// NB * TR + 2 rows; when a band is a whole image, the NB bands are NB
// images, each with its own Ho + 2 window rows.  Window cells are 64 bytes
// (one slice of one pixel), chunks swizzled as in conv_halo.hip; cells
// outside the image hold zp_x' and image cells are legalised once, after
// the loads land, so the nine taps are plain shifted LDS reads.
#include "conv_common.h"

namespace qnn {

using namespace conv;

namespace {

template <int N>
__device__ __forceinline__ void wait_vm()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
    asm volatile("" ::: "memory");
}

__device__ __forceinline__ int cell_swz(int q)
{
    return (q >> 2) & 3;
}

struct WinGeom {
    int tr;        // output rows per band
    int bands;     // bands per image
    int whole;     // 1: a band is a whole image, the NB bands are NB images
    int srows;     // window rows per band slot in whole-image mode: Ho + 2
    int hr, hc;    // window rows (all slots) and columns: Wo + 2
    int ninst;     // 1 KB loads per slice of the window
    int wbytes;    // window bytes (every slice)
    int gpi;       // workgroups per image (shared mode)
    int ngrp;      // workgroups per channel tile
    int cch;       // 64-channel slices: C / 64
    int ngroups;   // slice groups: ceil(cch / KS)
    int gbytes;    // LDS bytes of one weight group: TCB * KS * 9 KB
    int jsteps;    // K-steps per 16-row block of the operand-order weights
};

constexpr int kTaps = 9;   // 3 x 3

struct WinCfg {
    int nb, ks, tcb;   // bands, reduction split, 16-channel blocks per workgroup
};
// configurations instantiated (index = the plan's tile number)
constexpr WinCfg kWinCfg[] = {
    {4, 2, 2}, {2, 2, 2}, {4, 1, 2}, {8, 1, 2},
};
constexpr int kWinCount = sizeof(kWinCfg) / sizeof(kWinCfg[0]);

constexpr int stage_pitch(int tcb)
{
    return tcb * 16 + 16;
}

bool win_geometry(const ConvArgs &a, int cfg, WinGeom *g)
{
    if (cfg < 0 || cfg >= kWinCount)
        return false;
    const WinCfg c = kWinCfg[cfg];
    if (a.R != 3 || a.S != 3 || a.sh != 1 || a.sw != 1 || a.dh != 1 || a.dw != 1 || a.C % 64 != 0 || a.Wo < 1 ||
        a.Wo > 64 || a.Ho < 1 || a.rowpack || a.J != 9 * a.C || a.Jpad % 64 != 0 || a.Kpad % (16 * c.tcb) != 0)
        return false;
    if ((long long)a.N * a.H * a.W * a.C >= (1LL << 31))
        return false;
    g->tr = a.Ho < 64 / a.Wo ? a.Ho : 64 / a.Wo;
    g->bands = (a.Ho + g->tr - 1) / g->tr;
    g->whole = g->bands == 1;
    g->hc = a.Wo + 2;
    if (g->whole) {
        g->srows = a.Ho + 2;
        g->hr = c.nb * g->srows;
        g->gpi = 0;
        g->ngrp = (a.N + c.nb - 1) / c.nb;
    } else {
        const int nb = g->bands < c.nb ? g->bands : c.nb;
        g->srows = 0;
        g->hr = nb * g->tr + 2;
        g->gpi = (g->bands + c.nb - 1) / c.nb;
        if ((long long)a.N * g->gpi >= (1LL << 30))
            return false;
        g->ngrp = a.N * g->gpi;
    }
    g->ninst = (g->hr * g->hc + 15) / 16;
    const int nw = c.nb * c.ks;
    if ((g->ninst + nw - 1) / nw > 32)   // one mask bit per load of a wave
        return false;
    g->cch = a.C / 64;
    g->wbytes = g->cch * g->ninst * 1024;
    g->ngroups = (g->cch + c.ks - 1) / c.ks;
    g->gbytes = c.tcb * c.ks * kTaps * 1024;
    g->jsteps = a.Jpad / 64;
    const long long tiles_c = (a.K + 16 * c.tcb - 1) / (16 * c.tcb);
    if ((long long)g->ngrp * tiles_c >= (1LL << 31))
        return false;
    return true;
}

size_t win_lds(const WinGeom &g, const WinCfg &c)
{
    // weight groups (two), then the window; the partial sums and the
    // channel records reuse the weight groups, the staging tiles the window
    const size_t wgt = 2 * (size_t)g.gbytes;
    const size_t part = (size_t)c.nb * (c.ks - 1) * c.tcb * 4 * 1024 + 1024;
    const size_t stage = (size_t)c.nb * 64 * stage_pitch(c.tcb);
    return (wgt > part ? wgt : part) + ((size_t)g.wbytes > stage ? (size_t)g.wbytes : stage);
}

}  // namespace

template <int NB, int KS, int TCB, bool FLIP>
__global__ void __launch_bounds__(NB * KS * 64, 1) conv_window_kernel(ConvArgs a, WinGeom g)
{
    constexpr int NW = NB * KS;
    constexpr int TC = 16 * TCB;
    constexpr int SP = stage_pitch(TCB);
    extern __shared__ __attribute__((aligned(1024))) int8_t smem[];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave
    const int bs = wave / KS;   // band slot
    const int ks = wave % KS;   // part of the reduction
    const int lrow = lane & 15, lchk = lane >> 4;

    const int ct = blockIdx.x % a.tiles_c;
    const int pgrp = blockIdx.x / a.tiles_c;
    const int c0 = ct * TC;

    // this wave's band: image, first output row, valid pixels, window row
    int n, oh0, row0;
    bool tile_ok;
    if (g.whole) {
        n = pgrp * NB + bs;
        tile_ok = n < a.N;
        oh0 = 0;
        row0 = bs * g.srows;
    } else {
        n = pgrp / g.gpi;
        const int band = (pgrp - n * g.gpi) * NB + bs;
        tile_ok = band < g.bands;
        oh0 = (tile_ok ? band : 0) * g.tr;
        row0 = tile_ok ? bs * g.tr : 0;
    }
    const int nn = tile_ok ? n : 0;
    const int trv = min(g.tr, a.Ho - oh0);
    const int npx = tile_ok ? trv * a.Wo : 0;
    const int m0 = (nn * a.Ho + oh0) * a.Wo;

    // LDS: two weight groups (after the main loop: the partial sums, then
    // the channel records), the window (after the main loop: the staging
    // tiles)
    constexpr int kPartBytes = NB * (KS - 1) * TCB * 4 * 1024;
    const size_t wgt = 2 * (size_t)g.gbytes;
    int8_t *wbuf = smem;
    int8_t *recs = smem + kPartBytes;
    int8_t *win = smem + (wgt > (size_t)kPartBytes + 1024 ? wgt : (size_t)kPartBytes + 1024);

    const __amdgpu_buffer_rsrc_t rx =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.x, (short)0, a.N * a.H * a.W * a.C, kBufFlags);
    const __amdgpu_buffer_rsrc_t rw =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.wf, (short)0, a.Kpad * a.Jpad, kBufFlags);

    // weight group gi into buffer gi & 1: LDS fragment ((i * KS + k) * 9 + t)
    // holds 16-row block c0 / 16 + i of K-step t * cch + gi * KS + k (tap t,
    // slice gi * KS + k); slices past the last are not loaded (never read)
    auto load_group = [&](int gi) {
        int8_t *dst = wbuf + (gi & 1) * g.gbytes;
        for (int f = wave; f < TCB * KS * kTaps; f += NW) {
            const int t = f % kTaps;
            const int ik = f / kTaps;
            const int k = ik % KS, i = ik / KS;
            const int cc = gi * KS + k;
            if (cc >= g.cch)
                continue;
            const int src = ((c0 / 16 + i) * g.jsteps + t * g.cch + cc) * 1024;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (__attribute__((address_space(3))) void *)(dst + f * 1024),
                                                     16, lane * 16, src, 0, 0);
        }
    };

    load_group(0);

    // window: load k (of every slice) fills cells 16 k .. 16 k + 15 and is
    // issued by wave k % NW as its load u = k / NW
    uint32_t oob = 0;
    const int nmine = (g.ninst - wave + NW - 1) / NW;
    {
        const int ncell = g.hr * g.hc;
        for (int u = 0; u < nmine; ++u) {
            const int k = wave + u * NW;
            const int q = k * 16 + (lane >> 2);
            const int hrow = q / g.hc;
            const int iw = q - hrow * g.hc - a.pl;
            int wn, ih;
            if (g.whole) {
                const int slot = hrow / g.srows;
                wn = pgrp * NB + slot;
                ih = hrow - slot * g.srows - a.pt;
            } else {
                wn = n;
                ih = (pgrp - n * g.gpi) * NB * g.tr - a.pt + hrow;
            }
            const bool in = q < ncell && wn < a.N && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
            oob |= (in ? 0u : 1u) << u;
            const int voff = in ? ((wn * a.H + ih) * a.W + iw) * a.C + (((lane & 3) ^ cell_swz(q)) << 4) : kOutOfRange;
            for (int cc = 0; cc < g.cch; ++cc)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rx, (__attribute__((address_space(3))) void *)(win + (cc * g.ninst + k) * 1024), 16, voff, cc * 64,
                    0, 0);
        }
    }
    wait_vm<0>();
    // the window as x': each lane rewrites the 16 bytes it loaded (LDS
    // accesses of one wave run in order); the barrier publishes them
    {
        const v4i zp = v4i{(int)a.zp4, (int)a.zp4, (int)a.zp4, (int)a.zp4};
        const v4i fl = v4i{(int)0x80808080, (int)0x80808080, (int)0x80808080, (int)0x80808080};
        for (int cc = 0; cc < g.cch; ++cc) {
            int8_t *base = win + (cc * g.ninst + wave) * 1024 + lane * 16;
            for (int u0 = 0; u0 < nmine; u0 += 4) {
                v4i v[4];
#pragma unroll
                for (int d = 0; d < 4; ++d)
                    if (FLIP && u0 + d < nmine && !((oob >> (u0 + d)) & 1u))
                        v[d] = *(const v4i *)(base + (u0 + d) * NW * 1024);
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    if (u0 + d >= nmine)
                        continue;
                    const bool out = (oob >> (u0 + d)) & 1u;
                    if (out)
                        *(v4i *)(base + (u0 + d) * NW * 1024) = zp;
                    else if (FLIP)
                        *(v4i *)(base + (u0 + d) * NW * 1024) = v[d] ^ fl;
                }
            }
        }
    }

    // window sums of the band's pixels (term 3), used in the epilogue
    int s3j[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int p = j * 16 + lrow;
        s3j[j] = a.asum ? a.asum[p < npx ? m0 + p : 0] : 0;
    }

    // operand rows: pixel p = 16 j + lrow of the band is window cell
    // (row0 + p / Wo) * hc + p % Wo at tap (0, 0); pixels past the band read
    // a cell of the window and are never stored
    int qb[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        int p = j * 16 + lrow;
        p = p < npx ? p : 0;
        const int t = p / a.Wo;
        qb[j] = (row0 + t) * g.hc + (p - t * a.Wo);
    }

    // the accumulators of the ks = 0 waves start at bconst of their channels
    v4i acc[TCB][4];
#pragma unroll
    for (int i = 0; i < TCB; ++i) {
        v4i b0 = v4i{0, 0, 0, 0};
        if (ks == 0) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                b0[e] = a.chan[c0 + i * 16 + lchk * 4 + e].bconst;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = b0;
    }

    __syncthreads();   // the window and the first weight group are in LDS

    for (int gi = 0; gi < g.ngroups; ++gi) {
        if (gi > 0) {
            wait_vm<0>();      // this wave's share of group gi has landed
            __syncthreads();   // everyone's share, and group gi - 1 is no longer read
        }
        if (gi + 1 < g.ngroups)
            load_group(gi + 1);
        const int cc = gi * KS + ks;
        if (cc < g.cch) {
            const int8_t *wl = wbuf + (gi & 1) * g.gbytes + ks * kTaps * 1024 + lane * 16;
            const int8_t *hl = win + cc * g.ninst * 1024;
#pragma unroll
            for (int t = 0; t < kTaps; ++t) {
                const int toff = (t / 3) * g.hc + (t % 3);
                v4i A[TCB], B[4];
#pragma unroll
                for (int i = 0; i < TCB; ++i)
                    A[i] = *(const v4i *)(wl + (i * KS * kTaps + t) * 1024);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int q = qb[j] + toff;
                    B[j] = *(const v4i *)(hl + q * 64 + ((lchk ^ cell_swz(q)) << 4));
                }
#pragma unroll
                for (int i = 0; i < TCB; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A[i], B[j], acc[i][j], 0, 0, 0);
            }
        }
    }

    // ---- partial sums of a band's KS waves, channel records -------------------
    __syncthreads();   // every wave is past its last read of the weights and the window
    if (wave == NW - 1) {
        // records c0 .. c0 + 63 (those past Kpad read zeros and are not used)
        const __amdgpu_buffer_rsrc_t rc =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.chan, (short)0, a.Kpad * (int)sizeof(ChanRec), kBufFlags);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rc, (__attribute__((address_space(3))) void *)recs, 16,
                                                 (c0 + lane) * (int)sizeof(ChanRec), 0, 0, 0);
    }
    int32_t *part = (int32_t *)wbuf;
    if constexpr (KS > 1) {
        if (ks > 0) {
#pragma unroll
            for (int i = 0; i < TCB; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    *(v4i *)(part + ((((bs * (KS - 1) + ks - 1) * TCB + i) * 4 + j) * 64 + lane) * 4) = acc[i][j];
        }
    }
    wait_vm<0>();
    __syncthreads();   // partial sums and records are in LDS
    if constexpr (KS > 1) {
        if (ks > 0)
            return;
#pragma unroll
        for (int k = 1; k < KS; ++k)
#pragma unroll
            for (int i = 0; i < TCB; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] += *(const v4i *)(part + ((((bs * (KS - 1) + k - 1) * TCB + i) * 4 + j) * 64 + lane) * 4);
    }

    // ---- epilogue (the ks = 0 wave of each band) ------------------------------
    // block (i, j): channels c0 + 16 i + 4 lchk .. +3 of pixel m0 + 16 j + lrow;
    // the band's staging tile is in the window's space, its own
    int8_t *stage = win + bs * 64 * SP;
    const bool staged = a.staged && a.mode == OUT_REQUANT;
    v4i zw[TCB];
    if (a.asum) {
#pragma unroll
        for (int i = 0; i < TCB; ++i)
            zw[i] = *(const v4i *)(a.zpw + c0 + i * 16 + lchk * 4);
    }
#pragma unroll
    for (int i = 0; i < TCB; ++i) {
        const int ch = c0 + i * 16 + lchk * 4;
        v4i rec[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            rec[e] = *(const v4i *)(recs + (i * 16 + lchk * 4 + e) * (int)sizeof(ChanRec));
            rec[e].y = 0;   // bconst is already in the sums
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int p = j * 16 + lrow;
            const bool live = p < npx;
            const int m = m0 + p;
            v4i v = acc[i][j];
            if (a.asum)
                v -= zw[i] * v4i{s3j[j], s3j[j], s3j[j], s3j[j]};
            if (staged) {
                *(uint32_t *)(stage + p * SP + i * 16 + lchk * 4) = requant4(a, v, rec);
                continue;
            }
            if (!live || ch >= a.K)
                continue;
            const size_t off = (size_t)m * a.y_ldc + a.y_coff + ch;
            const bool full = a.vec_store && ch + 3 < a.K;
            if (a.mode == OUT_INT32) {
                int32_t *yp = (int32_t *)a.y + off;
                if (full) {
                    __builtin_nontemporal_store(v, (v4i *)yp);
                } else {
                    for (int e = 0; e < 4 && ch + e < a.K; ++e)
                        yp[e] = v[e];
                }
            } else {
                const uint32_t packed = requant4(a, v, rec);
                uint8_t *yp = (uint8_t *)a.y + off;
                if (full) {
                    __builtin_nontemporal_store(packed, (uint32_t *)yp);
                } else {
                    for (int e = 0; e < 4 && ch + e < a.K; ++e)
                        yp[e] = (uint8_t)(packed >> (8 * e));
                }
            }
        }
    }
    if (!staged)
        return;
    // copy out: 64 rows x TC / 16 chunks of 16 bytes
    const int kmax = a.K - c0;
#pragma unroll
    for (int k = 0; k < TCB; ++k) {
        const int idx = k * 64 + lane;
        const int pl = idx / TCB, qc = idx % TCB;
        if (pl >= npx || qc * 16 >= kmax)
            continue;
        const v4i v = *(const v4i *)(stage + pl * SP + qc * 16);
        uint8_t *dst = (uint8_t *)a.y + (size_t)(m0 + pl) * a.y_ldc + a.y_coff + c0 + qc * 16;
        if (qc * 16 + 16 <= kmax) {
            __builtin_nontemporal_store(v, (v4i *)dst);
        } else {
            for (int e = 0; e < kmax - qc * 16; ++e)
                dst[e] = (uint8_t)((uint32_t)v[e >> 2] >> (8 * (e & 3)));
        }
    }
}

int win_count()
{
    return kWinCount;
}

int win_channels(int cfg)
{
    return cfg >= 0 && cfg < kWinCount ? 16 * kWinCfg[cfg].tcb : 0;
}

int win_threads(int cfg)
{
    return cfg >= 0 && cfg < kWinCount ? 64 * kWinCfg[cfg].nb * kWinCfg[cfg].ks : 0;
}

size_t win_lds_bytes(const ConvArgs &a, int cfg)
{
    WinGeom g;
    if (!win_geometry(a, cfg, &g))
        return 0;
    return win_lds(g, kWinCfg[cfg]);
}

long long win_workgroups_per_ctile(const ConvArgs &a, int cfg)
{
    WinGeom g;
    if (!win_geometry(a, cfg, &g))
        return -1;
    return g.ngrp;
}

template <int CFG>
static hipError_t launch_win_cfg(const ConvArgs &a, const WinGeom &g, hipStream_t st)
{
    constexpr WinCfg c = kWinCfg[CFG];
    const size_t lds = win_lds(g, c);
    const dim3 grid((unsigned)(a.tiles_c * g.ngrp));
    const dim3 block(64 * c.nb * c.ks);
    if (a.flip4)
        launch_main((conv_window_kernel<c.nb, c.ks, c.tcb, true>), grid, block, lds, st, a, g);
    else
        launch_main((conv_window_kernel<c.nb, c.ks, c.tcb, false>), grid, block, lds, st, a, g);
    return hipGetLastError();
}

hipError_t launch_conv_window(const ConvArgs &a, int cfg, hipStream_t st)
{
    WinGeom g;
    if (!win_geometry(a, cfg, &g) || a.tiles_c != (a.K + win_channels(cfg) - 1) / win_channels(cfg))
        return hipErrorInvalidValue;
    switch (cfg) {
    case 0: return launch_win_cfg<0>(a, g, st);
    case 1: return launch_win_cfg<1>(a, g, st);
    case 2: return launch_win_cfg<2>(a, g, st);
    case 3: return launch_win_cfg<3>(a, g, st);

    default: return hipErrorInvalidValue;
    }
}

}  // namespace qnn
