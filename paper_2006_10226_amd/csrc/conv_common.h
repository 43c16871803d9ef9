// Device helpers shared by the implicit-GEMM conv kernels (conv_tap.hip,
// conv_dma.hip): LDS swizzle, fixed-point requantize, pixel decode and the
// tile epilogue.
#pragma once

#include "qnn_internal.h"

namespace qnn {

typedef int v4i __attribute__((ext_vector_type(4)));

namespace conv {

constexpr int kBufFlags = 0x00020000;   // raw buffer, 32-bit data format
constexpr int kOutOfRange = (int)0x80000000;

// Physical 16-byte chunk of logical chunk q in an LDS row of CPR chunks; it
// depends on row & 15 only.  Sixteen lanes reading rows 0..15 at one
// logical chunk hit 16 distinct 16-byte bank groups (rows of 128 bytes
// alternate between the two bank halves; rows of 64 bytes cycle through 4).
template <int CPR>
__device__ __forceinline__ int swz(int row)
{
    if constexpr (CPR == 8)
        return (row & 7) ^ ((row >> 3) & 1);
    else
        return ((row >> 1) & 3) ^ ((row >> 3) & 1);
}

// n / d for 0 <= n < 2^31 with a host-made magic pair (see make_divider):
// q = umulhi(n, mul) >> shift, or n itself for d == 1 (mul == 0).
__device__ __forceinline__ int fast_div(int n, uint32_t mul, uint32_t shift)
{
    return mul ? (int)(__umulhi((uint32_t)n, mul) >> shift) : n;
}

// Requantize four accumulators of consecutive channels (records rec[e] =
// {mult, bconst, rndzp, shift}) and pack the output bytes.  The 32-bit form
// (HALF_UP, 33 <= shift <= 53) is exact: with hi the signed high word of
// v * mult, floor((v*mult + 2^(shift-1)) / 2^shift) equals
// floor((hi + 2^(shift-33)) / 2^(shift-32)), and rndzp also carries
// (zp_y + off) * 2^(shift-32), off = 128 for int8 outputs, which the final
// XOR removes again.
__device__ __forceinline__ uint32_t requant4(const ConvArgs &a, v4i acc, const v4i (&rec)[4])
{
    uint32_t packed = 0;
    if (a.fast_rq) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int v = (int)((uint32_t)acc[e] + (uint32_t)rec[e].y);
            const int t = (__mulhi(v, rec[e].x) + rec[e].z) >> (rec[e].w & 31);   // shift - 32: shift is in [33, 53]
            packed |= (uint32_t)clamp_i32(t, a.lo_off, a.hi_off) << (8 * e);
        }
        return packed ^ a.out_xor;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int v = (int)((uint32_t)acc[e] + (uint32_t)rec[e].y);   // wraps exactly when the sum fits
        long long o = rounding_mul_shift(v, rec[e].x, rec[e].w, a.rounding) + a.zp_y;
        o = o < a.lo ? a.lo : (o > a.hi ? a.hi : o);
        packed |= ((uint32_t)o & 0xffu) << (8 * e);
    }
    return packed;
}

// Residual qnn.add fused into the epilogue.  The staged copy-out hands
// thread tid the 16-byte chunks idx = it * NT + tid (it < ITERS) of the
// tile: pixel row idx / CH, channels 16 * (idx % CH) on; the residual
// chunks of the same elements are loaded at the start of the epilogue
// (residual_prefetch), so that their memory latency overlaps the
// requantize and the staging.

// Whether the residual bytes of a chunk of n <= 16 channels come by one
// 16-byte load (residual rows 16-byte aligned, chunk whole); the copy-out
// loads the others byte by byte.
__device__ __forceinline__ bool residual_chunk_vec(const ConvArgs &a, int n)
{
    return a.res_vec && n == 16;
}

template <int TC, int TP, int NT>
__device__ __forceinline__ void residual_prefetch(const ConvArgs &a, int c0, int p0,
                                                  v4i (&r)[(TP * (TC / 16) + NT - 1) / NT])
{
    constexpr int CH = TC / 16, ITERS = (TP * CH + NT - 1) / NT;
    const int kmax = a.K - c0;
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
        const int idx = it * NT + (int)threadIdx.x;
        const int pl = idx / CH, qc = idx % CH;
        const int m = p0 + pl;
        r[it] = v4i{0, 0, 0, 0};
        if (idx < TP * CH && m < a.M && qc * 16 < kmax && residual_chunk_vec(a, min(16, kmax - qc * 16)))
            r[it] = __builtin_nontemporal_load(
                (const v4i *)(a.res + (size_t)m * a.r_ldc + a.r_coff + c0 + qc * 16));
    }
}

// The add of 16 requantized output bytes v (dtype ydt) and the residual
// bytes r of the same elements (rdt), through the add's own arithmetic;
// returns the sum's bytes.  One 4-byte word per pass, the words rotated
// through position 0 (a rolled loop keeps a single copy of add_one's code).
__device__ __forceinline__ v4i residual_add16(const ConvArgs &a, v4i v, v4i r)
{
    v4i o = v4i{0, 0, 0, 0};
#pragma unroll 1
    for (int q = 0; q < 4; ++q) {
        uint32_t ow = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t xb = ((uint32_t)v[0] >> (8 * e)) & 0xffu;
            const uint32_t rb = ((uint32_t)r[0] >> (8 * e)) & 0xffu;
            const int x = a.ydt == 1 ? (int)(int8_t)xb : (int)xb;
            const int y = a.rdt == 1 ? (int)(int8_t)rb : (int)rb;
            ow |= ((uint32_t)add_one(a.fadd, x, y) & 0xffu) << (8 * e);
        }
        o = v4i{o[1], o[2], o[3], (int)ow};
        v = v4i{v[1], v[2], v[3], v[0]};
        r = v4i{r[1], r[2], r[3], r[0]};
    }
    return o;
}

typedef __attribute__((address_space(3))) int32_t lds_i32;

// The add with the term tables in LDS (AddArgs::tab copied there): each
// element is clamp(tab[x] + tab[256 + r]).
__device__ __forceinline__ v4i residual_add16_tab(const ConvArgs &a, v4i v, v4i r, const lds_i32 *tab)
{
    v4i o;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        uint32_t ow = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t xb = ((uint32_t)v[w] >> (8 * e)) & 0xffu;
            const uint32_t rb = ((uint32_t)r[w] >> (8 * e)) & 0xffu;
            const int t = clamp_i32(tab[xb] + tab[256 + rb], a.fadd.lo, a.fadd.hi);
            ow |= ((uint32_t)t & 0xffu) << (8 * e);
        }
        o[w] = (int)ow;
    }
    return o;
}

// LDS home of the term tables in the fused instantiations.
template <bool FUSE>
__device__ __forceinline__ lds_i32 *fuse_tables()
{
    if constexpr (FUSE) {
        __shared__ __attribute__((aligned(16))) int32_t tab[512];
        return (lds_i32 *)tab;
    } else {
        return nullptr;
    }
}

// Copy-out of a staged tile (TP pixel rows of SP bytes in LDS, the tile's
// first min(TC, kmax) channels valid) with the residual add applied, the
// residual chunks prefetched in r (byte loads here where they were not);
// tab: the term tables in LDS, or nullptr for the add's own arithmetic.
template <int TC, int TP, int NT, int SP>
__device__ __forceinline__ void copy_out_residual(const ConvArgs &a, const int8_t *stage, int c0, int p0, int kmax,
                                                  const v4i (&r)[(TP * (TC / 16) + NT - 1) / NT],
                                                  const lds_i32 *tab)
{
    constexpr int CH = TC / 16, ITERS = (TP * CH + NT - 1) / NT;
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
        const int idx = it * NT + (int)threadIdx.x;
        const int pl = idx / CH, qc = idx % CH;
        const int m = p0 + pl;
        if (idx < TP * CH && m < a.M && qc * 16 < kmax) {
            const int n = min(16, kmax - qc * 16);
            v4i rv = r[it];
            if (!residual_chunk_vec(a, n)) {
                const uint8_t *rp = a.res + (size_t)m * a.r_ldc + a.r_coff + c0 + qc * 16;
                uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
                for (int e = 0; e < 16; ++e)
                    if (e < n)
                        w[e >> 2] |= (uint32_t)rp[e] << (8 * (e & 3));
                rv = v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
            }
            const v4i sv = *(const v4i *)(stage + pl * SP + qc * 16);
            const v4i v = tab ? residual_add16_tab(a, sv, rv, tab) : residual_add16(a, sv, rv);
            uint8_t *dst = (uint8_t *)a.y + (size_t)m * a.y_ldc + a.y_coff + c0 + qc * 16;
            if (n == 16) {
                __builtin_nontemporal_store(v, (v4i *)dst);
            } else {
#pragma unroll
                for (int e = 0; e < 16; ++e)
                    if (e < n)
                        dst[e] = (uint8_t)((uint32_t)v[e >> 2] >> (8 * (e & 3)));
            }
        }
    }
}

// 16-byte LDS read issued as inline assembly.  The compiler orders every LDS
// read it sees after all LDS-direct loads still in flight (it cannot tell
// which LDS bytes they write), which drains a ring of staged K-steps at
// every step; the kernels that read a ring this way order each read after
// the loads of its own stage themselves (vmcnt waits and barriers).  The
// result may be used only after lds_settle.
__device__ __forceinline__ v4i lds_read16(const int8_t *p)
{
    v4i r;
    const uint32_t addr = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) int8_t *)p;
    asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(addr) : "memory");
    return r;
}

// Waits until at most N of this wave's LDS reads (the N issued last) are in
// flight, then marks the given fragments as produced after the wait, so
// that no use of them is scheduled before it.
template <int N>
__device__ __forceinline__ void lds_wait()
{
    static_assert(N >= 0 && N <= 15, "lgkmcnt range");
    asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
}
template <int F>
__device__ __forceinline__ void lds_settled(v4i (&f)[F])
{
#pragma unroll
    for (int i = 0; i < F; ++i)
        asm volatile("" : "+v"(f[i]));
}

// One channel record of the tile's records in LDS, read through an LDS
// pointer (a generic pointer would make it a flat load, which also waits
// for every global load in flight).
__device__ __forceinline__ v4i lds_rec(const ChanRec *p)
{
    return *(const __attribute__((address_space(3))) v4i *)(const __attribute__((address_space(3))) void *)p;
}

// Adds bconst (bias and terms 2 and 4) of each block's four channels to the
// accumulators of a WC x WP wave grid, from the tile's records in LDS (the
// epilogue then leaves bconst out of the requantize).  ASYNC: the records
// are read with lds_read16 (the caller's waits cover their LDS-direct load).
template <int TC, int TP, int WC, int WP, bool ASYNC = false>
__device__ __forceinline__ void add_bconst(v4i (&acc)[TC / WC / 16][TP / WP / 16], const ChanRec *recs)
{
    constexpr int WTC = TC / WC, FC = WTC / 16, FP = TP / WP / 16;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wc = wave / WP;
    if constexpr (ASYNC) {
        v4i r[FC * 4];
#pragma unroll
        for (int i = 0; i < FC; ++i) {
            const int cl = wc * WTC + i * 16 + (lane >> 4) * 4;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                r[i * 4 + e] = lds_read16((const int8_t *)(recs + cl + e));
        }
        lds_wait<0>();
        lds_settled(r);
#pragma unroll
        for (int i = 0; i < FC; ++i) {
            const v4i b = v4i{r[i * 4][1], r[i * 4 + 1][1], r[i * 4 + 2][1], r[i * 4 + 3][1]};
#pragma unroll
            for (int j = 0; j < FP; ++j)
                acc[i][j] += b;
        }
    } else {
#pragma unroll
        for (int i = 0; i < FC; ++i) {
            const int cl = wc * WTC + i * 16 + (lane >> 4) * 4;
            const v4i b = v4i{lds_rec(recs + cl).y, lds_rec(recs + cl + 1).y, lds_rec(recs + cl + 2).y,
                              lds_rec(recs + cl + 3).y};
#pragma unroll
            for (int j = 0; j < FP; ++j)
                acc[i][j] += b;
        }
    }
}

// Epilogue of one TC x TP tile held by NT/64 waves in a WC x WP grid of
// (TC/WC) x (TP/WP) wave tiles of 16x16 MFMA blocks: lane holds channels
// ch..ch+3 (4 * (lane >> 4) inside a 16-block) of pixel lane & 15 inside a
// 16-block.  Adds the padding correction (when the gather read zeros for
// taps outside the image) and term 3, then requantizes and stores, through
// `stage` (LDS, at least TP * (TC + 16) bytes when a.staged) as whole
// 16-byte pixel-row chunks, or directly.  Every wave must be past its last
// read of `stage` before the call.  `recs` holds the tile's channel
// records (channels c0 .. c0 + TC - 1) in LDS, and the accumulators
// already hold bconst (see add_bconst).  FUSE: the staged copy-out applies the residual add (the
// host launches these instantiations only with a.res set and a.staged).
template <int TC, int TP, int WC, int WP, int STAGE_BYTES, bool FUSE = false>
__device__ __forceinline__ void store_tile(const ConvArgs &a, v4i (&acc)[TC / WC / 16][TP / WP / 16], int8_t *stage,
                                           int c0, int p0, const ChanRec *recs)
{
    constexpr int NT = WC * WP * 64;
    constexpr int WTC = TC / WC, WTP = TP / WP;
    constexpr int FC = WTC / 16, FP = WTP / 16;
    static_assert(!FUSE || WTC * WTP <= kFuseMaxWaveTile, "fused add: wave tiles of at most kFuseMaxWaveTile");
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave
    const int wc = wave / WP, wpos = wave % WP;
    const int lrow = lane & 15, lchk = lane >> 4;
    const int mb = p0 + wpos * WTP + lrow;
    v4i rres[FUSE ? (TP * (TC / 16) + NT - 1) / NT : 1];
    int32_t tabv[FUSE ? 512 / NT : 1];
    if constexpr (FUSE) {
        static_assert(512 % NT == 0, "the term tables split evenly over the threads");
        residual_prefetch<TC, TP, NT>(a, c0, p0, rres);
        if (a.fadd.tab) {
#pragma unroll
            for (int i = 0; i < 512 / NT; ++i)
                tabv[i] = a.fadd.tab[i * NT + tid];
        }
    }

    if (a.pcorr) {
        // taps outside the image were gathered as x = 0; the padding value
        // is zp_x, so add zp_x * (weights of those taps), per border class
#pragma unroll
        for (int j = 0; j < FP; ++j) {
            const int m = mb + j * 16;
            const int cls = m < a.M ? (int)a.pcls[m] : 255;
            if (cls != 255) {
#pragma unroll
                for (int i = 0; i < FC; ++i) {
                    const int ch = c0 + wc * WTC + i * 16 + lchk * 4;
                    acc[i][j] += *(const v4i *)(a.pcorr + (size_t)cls * a.Kpad + ch);
                }
            }
        }
    }
    if (a.asum) {
        // term 3 of Eq. (3): - zp_w[k] * (window sum of x~' at pixel m)
#pragma unroll
        for (int i = 0; i < FC; ++i) {
            const int ch = c0 + wc * WTC + i * 16 + lchk * 4;
            const v4i zw = *(const v4i *)(a.zpw + ch);
#pragma unroll
            for (int j = 0; j < FP; ++j) {
                const int s3 = a.asum[min(mb + j * 16, a.M - 1)];
                acc[i][j] -= zw * v4i{s3, s3, s3, s3};
            }
        }
    }
    if (a.staged) {
        constexpr int SP = (TP * (TC + 16) <= STAGE_BYTES) ? TC + 16 : TC;
        static_assert(TP * SP <= STAGE_BYTES, "output staging must fit the LDS buffers");
#pragma unroll
        for (int i = 0; i < FC; ++i) {
            const int cl = wc * WTC + i * 16 + lchk * 4;
            v4i rec[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
            {
                rec[e] = lds_rec(recs + cl + e);
                rec[e].y = 0;
            }
#pragma unroll
            for (int j = 0; j < FP; ++j) {
                const int pl = wpos * WTP + j * 16 + lrow;
                *(uint32_t *)(stage + pl * SP + cl) = requant4(a, acc[i][j], rec);
            }
        }
        if constexpr (FUSE) {
            if (a.fadd.tab) {
#pragma unroll
                for (int i = 0; i < 512 / NT; ++i)
                    fuse_tables<FUSE>()[i * NT + tid] = tabv[i];
            }
        }
        __syncthreads();
        constexpr int CH = TC / 16;
        const int kmax = a.K - c0;
        if constexpr (FUSE) {
            copy_out_residual<TC, TP, NT, SP>(a, stage, c0, p0, kmax, rres,
                                              a.fadd.tab ? fuse_tables<FUSE>() : nullptr);
            return;
        }
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
                        for (int e = 0; e < kmax - qc * 16; ++e)
                            dst[e] = (uint8_t)((uint32_t)v[e >> 2] >> (8 * (e & 3)));
                    }
                }
            }
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < FC; ++i) {
        const int ch = c0 + wc * WTC + i * 16 + lchk * 4;
        if (ch >= a.K)
            continue;
        const bool full = a.vec_store && ch + 3 < a.K;
        v4i rec[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
        {
            rec[e] = lds_rec(recs + (ch - c0) + e);
            rec[e].y = 0;
        }
#pragma unroll
        for (int j = 0; j < FP; ++j) {
            const int m = mb + j * 16;
            if (m >= a.M)
                continue;
            const size_t off = (size_t)m * a.y_ldc + a.y_coff + ch;
            if (a.mode == OUT_INT32) {
                int vals[4];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    vals[e] = (int)((uint32_t)acc[i][j][e] + (uint32_t)rec[e].y);
                int32_t *yp = (int32_t *)a.y + off;
                if (full) {
                    *(v4i *)yp = v4i{vals[0], vals[1], vals[2], vals[3]};
                } else {
                    for (int e = 0; e < 4 && ch + e < a.K; ++e)
                        yp[e] = vals[e];
                }
                continue;
            }
            const uint32_t packed = requant4(a, acc[i][j], rec);
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

}  // namespace conv
}  // namespace qnn
