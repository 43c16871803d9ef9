// Implicit-GEMM quantized conv2d / dense in which every wave works on its
// own 64 x 64 output tile (channels x pixels) and its own slice of the
// reduction, without barriers in the main loop.  For C % 64 == 0.
//
// Arithmetic as in conv_mfma.hip (Jain et al., Sec. II-B Eq. (3), Sec.
// III-B/C): term 1 on int8 MFMA over x' = x - 128 (uint8) or x (int8),
// terms 2 and 4 and the bias folded into ChanRec.bconst, term 3 from the
// window sums, requantize of Eq. (5) in the epilogue.
//
// Data path, per wave and K-step (64 bytes of the reduction, one filter tap
// because C % 64 == 0):
//   * weights: four 16 x 64 operand fragments, read straight into
//     registers from a copy of the packed weights laid out in MFMA operand
//     order (each fragment is one contiguous kilobyte, lane L's 16 bytes at
//     16 * L), so the loads are fully coalesced and need no LDS;
//   * activations: 64 pixels x 64 bytes gathered into the wave's private LDS
//     ring by LDS-direct buffer loads (four consecutive lanes read one
//     pixel's 64-byte run), then read back as four operand fragments.  Taps
//     outside the image read zeros (out-of-range offsets); the epilogue adds
//     the border-class correction as in conv_dma.hip.
// Waves never wait for each other while accumulating, so the latency of
// one wave's loads is covered by the other waves on its SIMD and by its own
// prefetch (activations and weights three stages ahead).  A workgroup of
// four waves covers 4 / KSPLIT tiles (eight waves, one tile, for KSPLIT =
// 8); with KSPLIT > 1 the waves of a tile take interleaved parts of the
// reduction and add their partial sums through LDS before the epilogue.
#include "conv_common.h"

#include <type_traits>

namespace qnn {

using namespace conv;

namespace {

// s_waitcnt on the vector-memory count only (gfx9 encoding), and on the
// LDS count only; each also fences the compiler's memory reordering.
template <int N>
__device__ __forceinline__ void wait_vm()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
    asm volatile("" ::: "memory");
}

__device__ __forceinline__ void wait_lgkm0()
{
    __builtin_amdgcn_s_waitcnt((15) | (7 << 4) | (0 << 8) | (3 << 14));
    asm volatile("" ::: "memory");
}

__device__ __forceinline__ int sw64w(int row)
{
    return (row >> 1) & 3;
}

}  // namespace

// Waves of a workgroup: four, or KSPLIT when a tile is split eight ways.
template <int KSPLIT>
constexpr int wave_count()
{
    return KSPLIT > 4 ? KSPLIT : 4;
}

template <int KSPLIT, int NS, bool FLIP>
__global__ void __launch_bounds__(wave_count<KSPLIT>() * 64, (KSPLIT > 4 ? 1 : 2)) conv_wave_kernel(ConvArgs a)
{
    constexpr int BK = 64;
    constexpr int NWV = wave_count<KSPLIT>();
    constexpr int TPW = NWV / KSPLIT;        // tiles per workgroup
    constexpr int BSTAGE = 64 * BK;          // activation bytes per stage and wave
    constexpr int RING = NS * BSTAGE;        // LDS ring of one wave
    constexpr int LPS = 8;                   // loads per lane per stage (4 weight, 4 activation)
    static_assert(NS == 4, "stage n + 3 reuses buffer (n - 1) mod 4");
    static_assert(KSPLIT == 1 || KSPLIT == 2 || KSPLIT == 4 || KSPLIT == 8, "split");
    // LDS: four wave rings; reused for the partial sums (4 x 16 KB) and the
    // output staging (TPW tiles of 64 pixels x 80 bytes)
    __shared__ __attribute__((aligned(1024))) int8_t lds[NWV * RING];
    // channel records of each tile of the workgroup, fetched at the start
    __shared__ __attribute__((aligned(16))) ChanRec wrec[TPW][64];
    static_assert(RING >= 64 * 64 * 4, "partial sums must fit");

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave
    const int tl = wave / KSPLIT;            // tile of this wave inside the workgroup
    const int ks_id = wave % KSPLIT;         // its part of the reduction

    // workgroups are dealt round-robin to the 8 XCDs; XCD x takes the x-th
    // eighth of the workgroup list
    const int nwg = (a.ntiles + TPW - 1) / TPW;
    const int chunk = (nwg + 7) >> 3;
    const int xcd = blockIdx.x & 7;
    const int wg = xcd * chunk + (blockIdx.x >> 3);
    if (wg >= min(nwg, (xcd + 1) * chunk))
        return;
    const int tile = wg * TPW + tl;
    const bool tile_ok = tile < a.ntiles;
    const int tt = tile_ok ? tile : 0;
    const int c0 = (tt % a.tiles_c) * 64;
    const int p0 = (tt / a.tiles_c) * 64;

    // reduction steps of this wave: ks = ks_id, ks_id + KSPLIT, ...
    const int nk = a.nk;
    const int my_steps = tile_ok ? (nk - ks_id + KSPLIT - 1) / KSPLIT : 0;

    const __amdgpu_buffer_rsrc_t rx =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.x, (short)0, a.N * a.H * a.W * a.C, kBufFlags);
    const __amdgpu_buffer_rsrc_t rw =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.wf, (short)0, a.Kpad * a.Jpad, kBufFlags);

    // weights in operand order: fragment (16-row block b, step s) at
    // ((b * Jsteps + s) * 64 + lane) * 16
    const int jsteps = a.Jpad / BK;
    const int wbase = ((c0 >> 4) * jsteps * 64 + lane) * 16;

    // activation gather: lane L fills row i * 16 + L / 4 of the 64-row block,
    // physical chunk L % 4, fetching logical chunk (L % 4) ^ sw64w(row)
    const int r16 = lane >> 2, pch = lane & 3;
    int pbase[4];
    uint32_t pmask[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = i * 16 + r16;
        const int m = p0 + row;
        pbase[i] = 0;
        pmask[i] = 0;
        if (tile_ok && m < a.M) {
            const int t = fast_div(m, a.mWo, a.sWo);
            const int ow = m - t * a.Wo;
            const int n = fast_div(t, a.mHo, a.sHo);
            const int oh = t - n * a.Ho;
            const int ih0 = oh * a.sh - a.pt, iw0 = ow * a.sw - a.pl;
            pbase[i] = ((n * a.H + ih0) * a.W + iw0) * a.C + ((pch ^ sw64w(row)) << 4);
            uint32_t rm = 0, cm = 0;
            for (int r = 0; r < a.R; ++r)
                rm |= (uint32_t)((unsigned)(ih0 + r * a.dh) < (unsigned)a.H) << r;
            for (int s = 0; s < a.S; ++s)
                cm |= (uint32_t)((unsigned)(iw0 + s * a.dw) < (unsigned)a.W) << s;
            pmask[i] = rm | (cm << 16);
        }
    }

    int8_t *ring = lds + wave * RING;
    const int cpt = a.C / BK;   // K-steps per filter tap
    // loader position of the activations: tap (lr, ls), channel offset lc
    int lr, ls, lc;
    {
        const int t = ks_id / cpt;
        lc = (ks_id - t * cpt) * BK;
        lr = t / a.S;
        ls = t - lr * a.S;
    }
    int voffB[4];
    auto set_tap = [&]() {
        const int toff = (lr * a.dh * a.W + ls * a.dw) * a.C;
        const uint32_t rin = lr < a.R ? 1u : 0u;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const bool v = (pmask[i] >> lr) & (pmask[i] >> (16 + ls)) & rin;
            voffB[i] = v ? pbase[i] + toff : kOutOfRange;
        }
    };
    // activations of this wave's n-th stage into its LDS ring, weights of
    // its n-th stage into registers (out of range past the end)
    auto issue_b = [&](int n) {
        const int oob = n < my_steps ? 0 : kOutOfRange;
        int8_t *dst = ring + (n & (NS - 1)) * BSTAGE;
        const int soffB = __builtin_amdgcn_readfirstlane(lc);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (__attribute__((address_space(3))) void *)(dst + i * 1024),
                                                     16, voffB[i] | oob, soffB, 0, 0);
        // advance KSPLIT steps
        lc += KSPLIT * BK;
        while (lc >= a.C) {
            lc -= a.C;
            if (++ls == a.S) {
                ls = 0;
                ++lr;
            }
        }
        set_tap();
    };
    auto load_a = [&](int n, v4i (&A)[4]) {
        const bool live = n < my_steps;
        const int soffA = live ? (ks_id + n * KSPLIT) * 1024 : 0;
        const int oob = live ? 0 : kOutOfRange;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            A[i] = __builtin_amdgcn_raw_buffer_load_b128(rw, (wbase + i * jsteps * 1024) | oob, soffA, 0);
    };

    // operand fragments of the activations: lane row lrow, chunk lchk
    const int lrow = lane & 15, lchk = lane >> 4;
    const int co = lrow * BK + ((lchk ^ sw64w(lrow)) << 4);
    // the first wave of each tile fetches the tile's 64 channel records into
    // LDS (the epilogue reads them after the loop's final barrier), and
    // starts its sums at bconst; the other waves of a split start at 0
    if (ks_id == 0) {
        const __amdgpu_buffer_rsrc_t rc =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.chan, (short)0, a.Kpad * (int)sizeof(ChanRec), kBufFlags);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rc, (__attribute__((address_space(3))) void *)wrec[tl], 16,
                                                 (c0 + lane) * (int)sizeof(ChanRec), 0, 0, 0);
    }
    v4i acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v4i b0 = v4i{0, 0, 0, 0};
        if (ks_id == 0) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                b0[e] = a.chan[c0 + i * 16 + lchk * 4 + e].bconst;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = b0;
    }
    auto step = [&](int n, v4i (&A)[4]) {
        const int8_t *src = ring + (n & (NS - 1)) * BSTAGE + co;
        // lds_read16: the wait for stage n above orders these reads after its
        // LDS-direct loads; the compiler would wait for every stage in flight
        v4i fb[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            fb[j] = lds_read16(src + j * 16 * BK);
        lds_wait<0>();
        lds_settled(fb);
        if constexpr (FLIP) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                fb[j] ^= v4i{(int)0x80808080, (int)0x80808080, (int)0x80808080, (int)0x80808080};
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A[i], fb[j], acc[i][j], 0, 0, 0);
    };

    // ---- main loop ---------------------------------------------------------
    // Activations run three stages ahead through the LDS ring and weights
    // three stages ahead through four register sets, issued interleaved
    // (activations of stage s, then its weights).  Step n first issues stage
    // n + 3, then waits until only the 24 loads of stages n + 1 .. n + 3 are
    // outstanding, i.e. stage n has landed, and until its LDS reads of stage
    // n - 1 have returned (that buffer is the one stage n + 3 overwrites).
    v4i A[4][4];
    set_tap();
    issue_b(0);
    load_a(0, A[0]);
    issue_b(1);
    load_a(1, A[1]);
    issue_b(2);
    load_a(2, A[2]);
    auto sub = [&](int n, auto K) __attribute__((always_inline)) {
        constexpr int k = decltype(K)::value;
        wait_lgkm0();
        issue_b(n + 3);
        load_a(n + 3, A[(k + 3) & 3]);
        wait_vm<3 * LPS>();
        step(n, A[k]);
    };
    int n = 0;
    for (; n + 4 <= my_steps; n += 4) {
        sub(n, std::integral_constant<int, 0>{});
        sub(n + 1, std::integral_constant<int, 1>{});
        sub(n + 2, std::integral_constant<int, 2>{});
        sub(n + 3, std::integral_constant<int, 3>{});
    }
    // 1 to 3 remaining steps: their weights are in sets 0, 1, 2
    if (n < my_steps)
        sub(n, std::integral_constant<int, 0>{});
    if (n + 1 < my_steps)
        sub(n + 1, std::integral_constant<int, 1>{});
    if (n + 2 < my_steps)
        sub(n + 2, std::integral_constant<int, 2>{});
    wait_vm<0>();   // trailing out-of-range loads write the ring too
    __syncthreads();

    // ---- partial sums of a tile's waves (KSPLIT > 1) ----------------------
    // wave (tl, s) keeps blocks blk = i * 4 + j with blk % KSPLIT == s
    int32_t *part = (int32_t *)lds;
    if constexpr (KSPLIT > 1) {
#pragma unroll
        for (int b = 0; b < 16; ++b)
            *(v4i *)(part + ((wave * 16 + b) * 64 + lane) * 4) = acc[b >> 2][b & 3];
        __syncthreads();
#pragma unroll
        for (int b = 0; b < 16; ++b) {
            if (b % KSPLIT != ks_id)
                continue;
            v4i s = v4i{0, 0, 0, 0};
#pragma unroll
            for (int w = 0; w < KSPLIT; ++w)
                s += *(const v4i *)(part + (((tl * KSPLIT + w) * 16 + b) * 64 + lane) * 4);
            acc[b >> 2][b & 3] = s;
        }
        __syncthreads();
    }

    // ---- epilogue ------------------------------------------------------------
    // block (i, j): channels c0 + 16 i + 4 lchk .. +3 of pixel p0 + 16 j + lrow
    constexpr int SP = 80;   // staging row: 64 channels + pad
    int8_t *stage = lds + tl * 64 * SP;
    const bool staged = a.staged && a.mode == OUT_REQUANT;
#pragma unroll
    for (int b = 0; b < 16; ++b) {
        if (b % KSPLIT != ks_id)
            continue;
        const int i = b >> 2, j = b & 3;
        const int ch = c0 + i * 16 + lchk * 4;
        const int m = p0 + j * 16 + lrow;
        v4i v = acc[i][j];
        if (a.pcorr && m < a.M) {
            const int cls = (int)a.pcls[m];
            if (cls != 255)
                v += *(const v4i *)(a.pcorr + (size_t)cls * a.Kpad + ch);
        }
        if (a.asum) {
            const int s3 = a.asum[min(m, a.M - 1)];
            v -= *(const v4i *)(a.zpw + ch) * v4i{s3, s3, s3, s3};
        }
        v4i rec[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
        {
            rec[e] = *(const v4i *)(wrec[tl] + (ch - c0) + e);
            rec[e].y = 0;   // bconst is in the sums already
        }
        if (staged) {
            *(uint32_t *)(stage + (j * 16 + lrow) * SP + i * 16 + lchk * 4) = requant4(a, v, rec);
            continue;
        }
        if (!tile_ok || m >= a.M || ch >= a.K)
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
    __syncthreads();
    // copy out: the KSPLIT waves of a tile share its 64 rows x 4 chunks
    const int kmax = a.K - c0;
    for (int idx = ks_id * 64 + lane; idx < 256; idx += KSPLIT * 64) {
        const int pl = idx >> 2, qc = idx & 3;
        const int m = p0 + pl;
        if (!tile_ok || m >= a.M || qc * 16 >= kmax)
            continue;
        const v4i v = *(const v4i *)(stage + pl * SP + qc * 16);
        uint8_t *dst = (uint8_t *)a.y + (size_t)m * a.y_ldc + a.y_coff + c0 + qc * 16;
        if (qc * 16 + 16 <= kmax) {
            __builtin_nontemporal_store(v, (v4i *)dst);
        } else {
            for (int e = 0; e < kmax - qc * 16; ++e)
                dst[e] = (uint8_t)((uint32_t)v[e >> 2] >> (8 * (e & 3)));
        }
    }
}

// Weights in MFMA operand order: out[((b * S + s) * 64 + L) * 16 + t] =
// wp[(16 b + L % 16) * Jpad + 64 s + 16 (L / 16) + t], S = Jpad / 64.
__global__ void __launch_bounds__(256) frag_pack_kernel(const int8_t *wp, int Kpad, int Jpad, int8_t *out)
{
    const long long n16 = (long long)Kpad * Jpad / 16;
    const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= n16)
        return;
    const int S = Jpad / 64;
    const int L = (int)(g & 63);
    const long long bs = g >> 6;
    const int s = (int)(bs % S);
    const int b = (int)(bs / S);
    const int8_t *src = wp + (size_t)(16 * b + (L & 15)) * Jpad + 64 * s + 16 * (L >> 4);
    *(v4i *)(out + g * 16) = *(const v4i *)src;
}

hipError_t launch_frag_pack(const int8_t *wp, int Kpad, int Jpad, int8_t *out, hipStream_t st)
{
    const long long n16 = (long long)Kpad * Jpad / 16;
    hipLaunchKernelGGL(frag_pack_kernel, dim3((unsigned)((n16 + 255) / 256)), dim3(256), 0, st, wp, Kpad, Jpad, out);
    return hipGetLastError();
}

int wave_tiles_per_block(int split)
{
    return split > 4 ? 1 : 4 / split;
}

int wave_threads(int split)
{
    return (split > 4 ? split : 4) * 64;
}

template <int KSPLIT>
static hipError_t launch_wave_split(const ConvArgs &a, hipStream_t st)
{
    constexpr int TPW = wave_count<KSPLIT>() / KSPLIT;
    const int nwg = (a.ntiles + TPW - 1) / TPW;
    const int grid = (nwg + 7) / 8 * 8;
    const dim3 block(wave_count<KSPLIT>() * 64);
    if (a.flip4)
        launch_main((conv_wave_kernel<KSPLIT, 4, true>), dim3(grid), block, 0, st, a);
    else
        launch_main((conv_wave_kernel<KSPLIT, 4, false>), dim3(grid), block, 0, st, a);
    return hipGetLastError();
}

hipError_t launch_conv_wave(const ConvArgs &a, int split, hipStream_t st)
{
    switch (split) {
    case 1: return launch_wave_split<1>(a, st);
    case 2: return launch_wave_split<2>(a, st);
    case 4: return launch_wave_split<4>(a, st);
    case 8: return launch_wave_split<8>(a, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace qnn
