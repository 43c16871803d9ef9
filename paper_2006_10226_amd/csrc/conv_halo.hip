// Implicit-GEMM quantized conv2d for stride-1, undilated 3x3 filters with
// C % 64 == 0 and output rows of at most 64 pixels.  Every wave computes
// whole output rows of one image (a band of at most 64 pixels) for 64
// output channels; the waves of a workgroup take consecutive bands of one
// image and share one LDS copy of their input window, and the workgroup's
// weights for the 64 channels are loaded once into LDS.
//
// Arithmetic as in conv_mfma.hip (Jain et al., Sec. II-B Eq. (3), Sec.
// III-B/C): term 1 on int8 MFMA over x' = x - 128 (uint8) or x (int8),
// terms 2 and 4 and the bias folded into ChanRec.bconst, term 3 from the
// window sums, requantize of Eq. (5) in the epilogue.
//
// Data path.  The tap walk of conv_dma.hip / conv_wave.hip fetches every
// input byte once per filter tap (nine times for 3x3) and every weight once
// per tile through the vector memory path.  Here a wave fetches its window
// of (NW * TR + 2) x (Wo + 2) pixels once (LDS-direct buffer loads, the
// waves taking turns) and fills the cells outside the image with zp_x'
// (held as zp_x' XOR 0x80 for uint8, because every fragment is legalised
// with one XOR after it is read; the XORs issue beside the MFMAs).
// The nine taps are nine shifted LDS views of the window: for output pixel
// (t, w) of the tile and tap (r, s) the operand row is window cell
// (t + r, w + s).  The accumulators start at the per-channel constant
// (bias and terms 2 and 4), so the epilogue only requantizes.
// A cell is 64 bytes (one 64-channel slice); its four 16-byte chunks are
// XOR-swizzled by (cell / 4) % 4 so that sixteen lanes reading sixteen
// consecutive cells at one logical chunk hit distinct bank groups.
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

// Tile geometry of one launch (host-computed).
struct HaloGeom {
    int tr;       // output rows per wave tile (a band)
    int hr, hc;   // window rows and columns: NW * tr + R - 1, Wo + S - 1
    int ninst;    // 1 KB loads per 64-channel slice of the window
    int wbytes;   // LDS bytes of the window (every slice)
    int bands;    // bands per image: ceil(Ho / tr)
    int gpi;      // workgroups per image and channel tile: ceil(bands / NW)
    int nst;      // K-steps of the filter: R * S * C / 64
    int jsteps;   // K-steps per 16-row block of the operand-order weights: Jpad / 64
    int nwg_p;    // workgroups per 64-channel tile: N * gpi
    int sep;      // 1: the staging tiles have LDS of their own (no barrier before the epilogue)
};

constexpr int kHaloR = 3, kHaloS = 3;
constexpr int kStagePitch = 80;   // staging row: 64 output bytes + pad
constexpr size_t kLdsPerCu = 160 * 1024;

bool halo_geometry(const ConvArgs &a, int nw, HaloGeom *g)
{
    if (a.R != kHaloR || a.S != kHaloS || a.sh != 1 || a.sw != 1 || a.dh != 1 || a.dw != 1 || a.C % 64 != 0 ||
        a.Wo < 1 || a.Wo > 64 || a.Ho < 1 || a.rowpack || (nw != 4 && nw != 8) || a.J != a.R * a.S * a.C ||
        a.Jpad % 64 != 0 || a.Kpad % 64 != 0)
        return false;
    if ((long long)a.N * a.H * a.W * a.C >= (1LL << 31))
        return false;
    g->tr = a.Ho < 64 / a.Wo ? a.Ho : 64 / a.Wo;
    g->bands = (a.Ho + g->tr - 1) / g->tr;
    // a workgroup never has more waves with a band than the image has bands
    const int nb = g->bands < nw ? g->bands : nw;
    g->hr = nb * g->tr + a.R - 1;
    g->hc = a.Wo + a.S - 1;
    g->ninst = (g->hr * g->hc + 15) / 16;
    if ((g->ninst + nw - 1) / nw > 32)   // one bit per load of a wave in the kernel's mask
        return false;
    const int cch = a.C / 64;
    g->wbytes = cch * g->ninst * 1024;
    g->gpi = (g->bands + nw - 1) / nw;
    g->nst = a.R * a.S * cch;
    g->jsteps = a.Jpad / 64;
    const long long nwg_p = (long long)a.N * g->gpi;
    if (nwg_p * ((a.K + 63) / 64) >= (1LL << 31))
        return false;
    g->nwg_p = (int)nwg_p;
    // separate staging space when it keeps the occupancy the launch bounds
    // ask for (one 8-wave or two 4-wave workgroups per CU)
    const size_t stage = (size_t)nw * 64 * kStagePitch;
    const size_t base = (size_t)g->nst * 4096 + 1024 + (size_t)g->wbytes;
    g->sep = base + stage <= (nw == 8 ? kLdsPerCu : kLdsPerCu / 2) ? 1 : 0;
    return true;
}

}  // namespace

template <int NW, bool FLIP>
__global__ void __launch_bounds__(NW * 64, NW == 4 ? 2 : 1) conv_halo_kernel(ConvArgs a, HaloGeom g)
{
    extern __shared__ __attribute__((aligned(1024))) int8_t smem[];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave

    // workgroup: one 64-channel tile and NW consecutive bands of one image
    const int ct = blockIdx.x % a.tiles_c;
    const int pg = blockIdx.x / a.tiles_c;
    const int c0 = ct * 64;
    const int n = pg / g.gpi;
    const int grp = pg - n * g.gpi;
    const int band = grp * NW + wave;
    const bool tile_ok = band < g.bands;
    const int oh0 = (tile_ok ? band : 0) * g.tr;
    const int trv = min(g.tr, a.Ho - oh0);
    const int npx = tile_ok ? trv * a.Wo : 0;   // valid output pixels of the tile
    const int m0 = (n * a.Ho + oh0) * a.Wo;     // they are m0 .. m0 + npx - 1
    const int cch = a.C >> 6;

    const __amdgpu_buffer_rsrc_t rx =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.x, (short)0, a.N * a.H * a.W * a.C, kBufFlags);
    const __amdgpu_buffer_rsrc_t rw =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.wf, (short)0, a.Kpad * a.Jpad, kBufFlags);

    // LDS: weights [4][nst] fragments of 1 KB, the 64 channel records, the
    // window, then one staging tile per wave (g.sep), else the staging tiles
    // reuse the window's space after the main loop
    int8_t *wts = smem;
    int8_t *recs = smem + g.nst * 4096;
    int8_t *win = recs + 1024;
    int8_t *stage = win + (g.sep ? g.wbytes : 0) + wave * (64 * kStagePitch);

    uint32_t oob = 0;   // bit u: this lane's cell of the wave's load u is outside the image
    // window: load k (of every slice cc) fills cells 16 k .. 16 k + 15 and is
    // issued by wave k % NW as its load u = k / NW; lane L fetches physical
    // chunk L % 4 of cell 16 k + L / 4, i.e. logical chunk (L % 4) ^ swizzle
    const int nmine = (g.ninst - wave + NW - 1) / NW;   // loads of this wave
    {
        const int ncell = g.hr * g.hc;
        const int ih0 = grp * NW * g.tr - a.pt, iw0 = -a.pl;
        for (int u = 0; u < nmine; ++u) {
            const int k = wave + u * NW;
            const int q = k * 16 + (lane >> 2);
            const int hr = q / g.hc;
            const int ih = ih0 + hr, iw = iw0 + (q - hr * g.hc);
            const bool in = q < ncell && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
            oob |= (in ? 0u : 1u) << u;
            const int voff = in ? ((n * a.H + ih) * a.W + iw) * a.C + (((lane & 3) ^ cell_swz(q)) << 4) : kOutOfRange;
            for (int cc = 0; cc < cch; ++cc)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rx, (__attribute__((address_space(3))) void *)(win + (cc * g.ninst + k) * 1024), 16, voff, cc * 64,
                    0, 0);
        }
    }
    // weights, after the window (its loads go to HBM, these mostly hit the
    // L2), in MFMA operand order: fragment (16-row block b, step s) of the
    // packed copy is the kilobyte at (b * jsteps + s) * 1024; LDS fragment
    // f = i * nst + st holds block c0 / 16 + i, step st
    for (int f = wave; f < 4 * g.nst; f += NW) {
        const int i = f / g.nst;
        const int st = f - i * g.nst;
        const int src = ((c0 / 16 + i) * g.jsteps + st) * 1024;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (__attribute__((address_space(3))) void *)(wts + f * 1024), 16,
                                                 lane * 16, src, 0, 0);
    }

    if (wave == NW - 1) {
        const __amdgpu_buffer_rsrc_t rc =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.chan, (short)0, a.Kpad * (int)sizeof(ChanRec), kBufFlags);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rc, (__attribute__((address_space(3))) void *)recs, 16,
                                                 (c0 + lane) * (int)sizeof(ChanRec), 0, 0, 0);
    }

    wait_vm<0>();

    // padding cells: each lane overwrites the 16 bytes of its loads that fell
    // outside the image (LDS accesses of one wave run in order; the barrier
    // below publishes them) with zp_x' in the stored form of the window,
    // which is x' XOR 0x80 for uint8 (the fragments are legalised with one
    // XOR after they are read)
    {
        const int zs = (int)(a.zp4 ^ (FLIP ? 0x80808080u : 0u));
        const v4i zp = v4i{zs, zs, zs, zs};
        for (int cc = 0; cc < cch; ++cc) {
            int8_t *base = win + (cc * g.ninst + wave) * 1024 + lane * 16;
            for (int u = 0; u < nmine; ++u)
                if ((oob >> u) & 1u)
                    *(v4i *)(base + u * NW * 1024) = zp;
        }
    }
    __syncthreads();   // every wave's share of the weights and records has landed

    // window sums of the tile's pixels (term 3), fetched now, used after
    // the main loop
    const int lrow0 = lane & 15;
    int s3j[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int p = j * 16 + lrow0;
        s3j[j] = a.asum ? a.asum[p < npx ? m0 + p : 0] : 0;
    }

    // operand rows: pixel p = 16 j + lrow of the tile is window cell
    // (wave * tr + p / Wo) * hc + p % Wo at tap (0, 0); pixels past the tile
    // (and every pixel of a wave without a band) read a cell of the window
    // and are never stored
    const int lrow = lane & 15, lchk = lane >> 4;
    int qb[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        int p = j * 16 + lrow;
        p = p < npx ? p : 0;
        const int t = p / a.Wo;
        qb[j] = ((tile_ok ? wave * g.tr : 0) + t) * g.hc + (p - t * a.Wo);
    }
    // accumulators start at bconst of their four channels
    v4i acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v4i b0;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            b0[e] = ((const v4i *)(recs + (i * 16 + lchk * 4 + e) * (int)sizeof(ChanRec)))->y;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = b0;
    }

    // the operands of tap t + 1 are read while the MFMAs of tap t run
    const int8_t *wl = wts + lane * 16;
    auto load_tap = [&](const int8_t *hl, int cc, int t, v4i (&A)[4], v4i (&B)[4]) __attribute__((always_inline)) {
        const int r = t / kHaloS, s = t - r * kHaloS;
        const int st = t * cch + cc;   // K-step of tap (r, s), slice cc
        const int toff = r * g.hc + s;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            A[i] = *(const v4i *)(wl + (i * g.nst + st) * 1024);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int q = qb[j] + toff;
            B[j] = *(const v4i *)(hl + q * 64 + ((lchk ^ cell_swz(q)) << 4));
        }
    };
    auto legalise = [&](v4i (&B)[4]) __attribute__((always_inline)) {
        if constexpr (FLIP) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                B[j] ^= v4i{(int)0x80808080, (int)0x80808080, (int)0x80808080, (int)0x80808080};
        }
    };
    for (int cc = 0; cc < cch; ++cc) {
        const int8_t *hl = win + cc * g.ninst * 1024;
        v4i A[2][4], B[2][4];
        load_tap(hl, cc, 0, A[0], B[0]);
#pragma unroll
        for (int t = 0; t < kHaloR * kHaloS; ++t) {
            if (t + 1 < kHaloR * kHaloS)
                load_tap(hl, cc, t + 1, A[(t + 1) & 1], B[(t + 1) & 1]);
            // keep the order: the reads of tap t + 1 are issued before the
            // MFMAs of tap t (the scheduler otherwise moves each read next
            // to its first use and waits on it there)
            __builtin_amdgcn_sched_barrier(0);
            legalise(B[t & 1]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A[t & 1][i], B[t & 1][j], acc[i][j], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
    }

    // ---- epilogue ------------------------------------------------------------
    // block (i, j): channels c0 + 16 i + 4 lchk .. +3 of pixel m0 + 16 j + lrow.
    // Staging tiles in the window's space overwrite it once every wave is
    // past its reads of it; a staging tile is one wave's own (LDS accesses
    // of one wave run in order).
    const bool staged = a.staged && a.mode == OUT_REQUANT;
    if (staged && !g.sep)
        __syncthreads();
    v4i zw[4];
    if (a.asum) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            zw[i] = *(const v4i *)(a.zpw + c0 + i * 16 + lchk * 4);
    }
    v4i rec[4];
#pragma unroll
    for (int b = 0; b < 16; ++b) {
        const int i = b >> 2, j = b & 3;
        const int ch = c0 + i * 16 + lchk * 4;
        const int p = j * 16 + lrow;
        const bool live = p < npx;
        const int m = m0 + p;
        v4i v = acc[i][j];
        if (a.asum)
            v -= zw[i] * v4i{s3j[j], s3j[j], s3j[j], s3j[j]};
        if (j == 0) {
            // records of the block row; bconst is already in the sums
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                rec[e] = *(const v4i *)(recs + (i * 16 + lchk * 4 + e) * (int)sizeof(ChanRec));
                rec[e].y = 0;
            }
        }
        if (staged) {
            *(uint32_t *)(stage + p * kStagePitch + i * 16 + lchk * 4) = requant4(a, v, rec);
            continue;
        }
        if (!live || ch >= a.K)
            continue;
        const size_t off = (size_t)m * a.y_ldc + a.y_coff + ch;
        const bool full = a.vec_store && ch + 3 < a.K;
        if (a.mode == OUT_INT32) {
            int vals[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                vals[e] = (int)((uint32_t)v[e] + (uint32_t)rec[e].y);
            int32_t *yp = (int32_t *)a.y + off;
            if (full) {
                *(v4i *)yp = v4i{vals[0], vals[1], vals[2], vals[3]};
            } else {
                for (int e = 0; e < 4 && ch + e < a.K; ++e)
                    yp[e] = vals[e];
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
    if (!staged)
        return;
    // copy out: 64 rows x 4 chunks of 16 bytes
    const int kmax = a.K - c0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int idx = k * 64 + lane;
        const int pl = idx >> 2, qc = idx & 3;
        if (pl >= npx || qc * 16 >= kmax)
            continue;
        const v4i v = *(const v4i *)(stage + pl * kStagePitch + qc * 16);
        uint8_t *dst = (uint8_t *)a.y + (size_t)(m0 + pl) * a.y_ldc + a.y_coff + c0 + qc * 16;
        if (qc * 16 + 16 <= kmax) {
            __builtin_nontemporal_store(v, (v4i *)dst);
        } else {
            for (int e = 0; e < kmax - qc * 16; ++e)
                dst[e] = (uint8_t)((uint32_t)v[e >> 2] >> (8 * (e & 3)));
        }
    }
}

size_t halo_lds_bytes(const ConvArgs &a, int nw)
{
    HaloGeom g;
    if (!halo_geometry(a, nw, &g))
        return 0;
    const size_t stage = (size_t)nw * 64 * kStagePitch;
    const size_t base = (size_t)g.nst * 4096 + 1024;
    return g.sep ? base + g.wbytes + stage : base + ((size_t)g.wbytes > stage ? (size_t)g.wbytes : stage);
}

int halo_layout(const ConvArgs &a, int nw)
{
    HaloGeom g;
    if (!halo_geometry(a, nw, &g))
        return -1;
    return g.sep;
}

long long halo_pixel_tiles(const ConvArgs &a)
{
    HaloGeom g;
    if (!halo_geometry(a, 4, &g))
        return -1;
    return (long long)a.N * g.bands;
}

template <int NW>
static hipError_t launch_halo_nw(const ConvArgs &a, const HaloGeom &g, hipStream_t st)
{
    const size_t lds = halo_lds_bytes(a, NW);
    const dim3 grid((unsigned)(a.tiles_c * g.nwg_p));
    if (a.flip4)
        launch_main((conv_halo_kernel<NW, true>), grid, dim3(NW * 64), lds, st, a, g);
    else
        launch_main((conv_halo_kernel<NW, false>), grid, dim3(NW * 64), lds, st, a, g);
    return hipGetLastError();
}

hipError_t launch_conv_halo(const ConvArgs &a, int nw, hipStream_t st)
{
    HaloGeom g;
    if (!halo_geometry(a, nw, &g) || a.tiles_c != (a.K + 63) / 64)
        return hipErrorInvalidValue;
    switch (nw) {
    case 4: return launch_halo_nw<4>(a, g, st);
    case 8: return launch_halo_nw<8>(a, g, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace qnn
