// Quantized 2-D pooling, Eq. (4) (Sec. III-B, QNN pooling): the input and
// output share one scale and zero point, so the kernel pools the quantized
// values directly and no requantize follows.
//
// Average: the window's cells are summed in int32 (the paper upcasts to
// int16 for its targets; int32 is exact for any window of up to 2^16 cells)
// and divided by the cell count with round to nearest, ties toward +inf
// (HALF_UP) or away from zero (HALF_AWAY).  Max: the largest in-input cell.
//
// One thread takes V consecutive channels (16, 4 or 1 bytes) of one output
// pixel; neighbouring threads take neighbouring channel groups, so each
// window cell is one coalesced row segment.  The kernel is bound by HBM
// traffic: every input byte once for non-overlapping windows (overlapping
// ones re-read from L2), every output byte once.
#include "qnn_internal.h"

namespace qnn {

// floor(num / den) for 0 <= num < 2^26 and 1 <= den <= 2^17 whose quotient is
// below 512: the float estimate is within 2^-14 of the quotient, so its
// truncation is off by at most one, which the exact integer remainder fixes
// (q * den < 2^27 is exact in the full-rate 24-bit multiply).
__device__ __forceinline__ int pool_div(int num, int den, float rcp)
{
    int q = (int)((float)num * rcp);
    const int r = num - (int)__umul24((unsigned)q, (unsigned)den);
    q += (r >= den) - (r < 0);
    return q;
}

template <int V>
__device__ __forceinline__ void pool_load(const int8_t *p, unsigned (&w)[(V + 3) / 4])
{
    if constexpr (V == 16) {
        const uint4 u = *(const uint4 *)p;
        w[0] = u.x; w[1] = u.y; w[2] = u.z; w[3] = u.w;
    } else if constexpr (V == 4) {
        w[0] = *(const unsigned *)p;
    } else {
        w[0] = (unsigned char)*p;
    }
}

// PACK (average, V >= 4, windows of at most 257 cells): bytes 0 and 2 of
// each loaded word are summed in the two 16-bit halves of one register,
// bytes 1 and 3 in another (int8 biased by +128 first); 257 * 255 < 2^16,
// so no half carries into the other.
// W3 (3x3 windows): the nine cells are loaded before any is used, so their
// memory latencies overlap (the loops of the general form wait once per
// window row, which is what small, latency-bound launches pay for); a cell
// outside the input reads the window's first cell inside it instead and
// is left out of the sum or maximum.
template <bool SIGNED, bool MAX, int V, bool PACK = false, bool W3 = false>
__global__ void __launch_bounds__(256) pool_kernel(PoolArgs a)
{
    constexpr int NW = (V + 3) / 4;
    const unsigned groups = (unsigned)(a.C / V);
    const long long total = (long long)a.N * a.Ho * a.Wo * groups;
    const long long step = (long long)gridDim.x * blockDim.x;
    for (long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x; gid < total; gid += step) {
        const unsigned u = (unsigned)gid;
        const unsigned g = u % groups;
        unsigned p = u / groups;
        const int ow = (int)(p % (unsigned)a.Wo);
        p /= (unsigned)a.Wo;
        const int oh = (int)(p % (unsigned)a.Ho);
        const int n = (int)(p / (unsigned)a.Ho);
        const int h0 = oh * a.sh - a.pt, w0 = ow * a.sw - a.pl;
        const int r0 = max(0, -h0), r1 = min(a.R, a.H - h0);
        const int s0 = max(0, -w0), s1 = min(a.S, a.W - w0);
        int acc[V];
#pragma unroll
        for (int i = 0; i < V; ++i)
            acc[i] = MAX ? (SIGNED ? -128 : 0) : 0;
        const int8_t *base = (const int8_t *)a.x + (size_t)n * a.H * a.W * a.C + (size_t)g * V;
        unsigned even[NW], odd[NW];
#pragma unroll
        for (int k = 0; k < NW; ++k)
            even[k] = odd[k] = 0;
        auto take = [&](const unsigned (&w)[NW]) {
            if constexpr (PACK) {
#pragma unroll
                for (int k = 0; k < NW; ++k) {
                    const unsigned x = SIGNED ? w[k] ^ 0x80808080u : w[k];
                    even[k] += x & 0x00ff00ffu;
                    odd[k] += (x >> 8) & 0x00ff00ffu;
                }
            } else {
#pragma unroll
                for (int i = 0; i < V; ++i) {
                    const unsigned b = (w[i / 4] >> (8 * (i % 4))) & 0xffu;
                    const int v = SIGNED ? (int)(signed char)b : (int)b;
                    acc[i] = MAX ? max(acc[i], v) : acc[i] + v;
                }
            }
        };
        if constexpr (W3) {
            if (r0 < r1 && s0 < s1) {
                unsigned w9[9][NW];
#pragma unroll
                for (int t = 0; t < 9; ++t) {
                    const int r = t / 3, c = t % 3;
                    const bool in = r >= r0 && r < r1 && c >= s0 && c < s1;
                    pool_load<V>(base + ((size_t)(h0 + (in ? r : r0)) * a.W + (w0 + (in ? c : s0))) * a.C, w9[t]);
                }
#pragma unroll
                for (int t = 0; t < 9; ++t) {
                    const int r = t / 3, c = t % 3;
                    if (r >= r0 && r < r1 && c >= s0 && c < s1)
                        take(w9[t]);
                }
            }
        } else {
        for (int r = r0; r < r1; ++r) {
            const int8_t *row = base + ((size_t)(h0 + r) * a.W + (w0 + s0)) * a.C;
            // unrolled so that several cells' loads are in flight at once
#pragma unroll 4
            for (int s = s0; s < s1; ++s, row += a.C) {
                unsigned w[NW];
                pool_load<V>(row, w);
                take(w);
            }
        }
        }
        if constexpr (PACK) {
            const int bias = SIGNED ? 128 * (r1 - r0) * (s1 - s0) : 0;
#pragma unroll
            for (int i = 0; i < V; ++i) {
                const unsigned h = (i % 2 == 0 ? even[i / 4] : odd[i / 4]) >> (16 * ((i % 4) / 2));
                acc[i] = (int)(h & 0xffffu) - bias;
            }
        }
        if constexpr (!MAX) {
            int cnt = (r1 - r0) * (s1 - s0);
            int pad_sum = 0;
            if (a.count_pad) {
                pad_sum = (a.R * a.S - cnt) * a.zp;
                cnt = a.R * a.S;
            }
            const int den = 2 * cnt;
            const float rcp = 1.0f / (float)den;
#pragma unroll
            for (int i = 0; i < V; ++i) {
                const int sum = acc[i] + pad_sum;
                if (!SIGNED) {
                    // sum >= 0: both roundings agree
                    acc[i] = pool_div(2 * sum + cnt, den, rcp);
                } else if (a.rounding == 1) {
                    const int m = pool_div(2 * abs(sum) + cnt, den, rcp);
                    acc[i] = sum < 0 ? -m : m;
                } else {
                    // sum >= -128 * cnt, so the shifted numerator is positive
                    acc[i] = pool_div(2 * sum + cnt + 128 * den, den, rcp) - 128;
                }
            }
        }
        unsigned o[NW];
#pragma unroll
        for (int k = 0; k < NW; ++k)
            o[k] = 0;
#pragma unroll
        for (int i = 0; i < V; ++i)
            o[i / 4] |= ((unsigned)acc[i] & 0xffu) << (8 * (i % 4));
        int8_t *dst = (int8_t *)a.y + (size_t)u * V;
        if constexpr (V == 16) {
            typedef unsigned u4 __attribute__((ext_vector_type(4)));
            __builtin_nontemporal_store(u4{o[0], o[1], o[2], o[3]}, (u4 *)dst);
        } else if constexpr (V == 4) {
            __builtin_nontemporal_store(o[0], (unsigned *)dst);
        } else {
            *dst = (int8_t)(o[0] & 0xffu);
        }
    }
}

// Few output pixels with large windows (global pooling): a workgroup of
// SPLIT_WAVES waves takes one output pixel and 64*V channels; wave k sums
// the window's cells k, k + SPLIT_WAVES, ... and the partial results meet
// in LDS, where wave 0 finishes them.  Every thread reaches the barrier.
constexpr int SPLIT_WAVES = 8;

template <bool SIGNED, bool MAX, int V>
__global__ void __launch_bounds__(64 * SPLIT_WAVES) pool_split_kernel(PoolArgs a, int chunks)
{
    __shared__ int part[SPLIT_WAVES][64 * V];
    const int lane = threadIdx.x % 64, wave = threadIdx.x / 64;
    const int chunk = blockIdx.x % chunks;
    const int p = blockIdx.x / chunks;
    const int ow = p % a.Wo, oh = (p / a.Wo) % a.Ho, n = p / (a.Wo * a.Ho);
    const int c0 = (chunk * 64 + lane) * V;
    const bool active = c0 < a.C;
    const int h0 = oh * a.sh - a.pt, w0 = ow * a.sw - a.pl;
    const int r0 = max(0, -h0), r1 = min(a.R, a.H - h0);
    const int s0 = max(0, -w0), s1 = min(a.S, a.W - w0);
    const int ws = s1 - s0, cells = (r1 - r0) * ws;
    int acc[V];
#pragma unroll
    for (int i = 0; i < V; ++i)
        acc[i] = MAX ? (SIGNED ? -128 : 0) : 0;
    if (active) {
        const int8_t *base = (const int8_t *)a.x + (size_t)n * a.H * a.W * a.C + c0;
#pragma unroll 4
        for (int idx = wave; idx < cells; idx += SPLIT_WAVES) {
            const int h = h0 + r0 + idx / ws, w = w0 + s0 + idx % ws;
            unsigned wd[(V + 3) / 4];
            pool_load<V>(base + ((size_t)h * a.W + w) * a.C, wd);
#pragma unroll
            for (int i = 0; i < V; ++i) {
                const unsigned b = (wd[i / 4] >> (8 * (i % 4))) & 0xffu;
                const int v = SIGNED ? (int)(signed char)b : (int)b;
                acc[i] = MAX ? max(acc[i], v) : acc[i] + v;
            }
        }
    }
#pragma unroll
    for (int i = 0; i < V; ++i)
        part[wave][lane * V + i] = acc[i];
    __syncthreads();
    if (wave != 0 || !active)
        return;
#pragma unroll
    for (int k = 1; k < SPLIT_WAVES; ++k)
#pragma unroll
        for (int i = 0; i < V; ++i)
            acc[i] = MAX ? max(acc[i], part[k][lane * V + i]) : acc[i] + part[k][lane * V + i];
    if constexpr (!MAX) {
        int cnt = cells, pad_sum = 0;
        if (a.count_pad) {
            pad_sum = (a.R * a.S - cnt) * a.zp;
            cnt = a.R * a.S;
        }
        const int den = 2 * cnt;
        const float rcp = 1.0f / (float)den;
#pragma unroll
        for (int i = 0; i < V; ++i) {
            const int sum = acc[i] + pad_sum;
            if (!SIGNED) {
                acc[i] = pool_div(2 * sum + cnt, den, rcp);
            } else if (a.rounding == 1) {
                const int m = pool_div(2 * abs(sum) + cnt, den, rcp);
                acc[i] = sum < 0 ? -m : m;
            } else {
                acc[i] = pool_div(2 * sum + cnt + 128 * den, den, rcp) - 128;
            }
        }
    }
    int8_t *dst = (int8_t *)a.y + (size_t)p * a.C + c0;
    unsigned o = 0;
#pragma unroll
    for (int i = 0; i < V; ++i)
        o |= ((unsigned)acc[i] & 0xffu) << (8 * i);
    if constexpr (V == 4)
        __builtin_nontemporal_store(o, (unsigned *)dst);
    else
        *dst = (int8_t)(o & 0xffu);
}

template <bool SIGNED, bool MAX>
static void launch_split_t(const PoolArgs &a, int vec, hipStream_t s)
{
    const int chunks = (a.C / vec + 63) / 64;
    const dim3 grid((unsigned)((long long)a.N * a.Ho * a.Wo * chunks));
    if (vec == 4) launch_main((pool_split_kernel<SIGNED, MAX, 4>), grid, dim3(64 * SPLIT_WAVES), 0, s, a, chunks);
    else launch_main((pool_split_kernel<SIGNED, MAX, 1>), grid, dim3(64 * SPLIT_WAVES), 0, s, a, chunks);
}

hipError_t launch_pool_split(const PoolArgs &a, bool is_signed, int vec, hipStream_t s)
{
    if ((long long)a.N * a.Ho * a.Wo == 0)
        return hipSuccess;
    const bool mx = a.mode == 1;
    if (is_signed) {
        if (mx) launch_split_t<true, true>(a, vec, s);
        else launch_split_t<true, false>(a, vec, s);
    } else {
        if (mx) launch_split_t<false, true>(a, vec, s);
        else launch_split_t<false, false>(a, vec, s);
    }
    return hipGetLastError();
}

template <bool SIGNED, bool MAX, bool W3>
static void launch_pool_w(const PoolArgs &a, int vec, dim3 grid, hipStream_t s)
{
    const bool pack = !MAX && (long long)a.R * a.S <= 257;
    if (vec == 16 && pack) launch_main((pool_kernel<SIGNED, MAX, 16, !MAX, W3>), grid, dim3(256), 0, s, a);
    else if (vec == 16) launch_main((pool_kernel<SIGNED, MAX, 16, false, W3>), grid, dim3(256), 0, s, a);
    else if (vec == 4 && pack) launch_main((pool_kernel<SIGNED, MAX, 4, !MAX, W3>), grid, dim3(256), 0, s, a);
    else if (vec == 4) launch_main((pool_kernel<SIGNED, MAX, 4, false, W3>), grid, dim3(256), 0, s, a);
    else launch_main((pool_kernel<SIGNED, MAX, 1, false, W3>), grid, dim3(256), 0, s, a);
}

template <bool SIGNED, bool MAX>
static void launch_pool_t(const PoolArgs &a, int vec, dim3 grid, hipStream_t s)
{
    if (a.R == 3 && a.S == 3)
        launch_pool_w<SIGNED, MAX, true>(a, vec, grid, s);
    else
        launch_pool_w<SIGNED, MAX, false>(a, vec, grid, s);
}

hipError_t launch_pool(const PoolArgs &a, bool is_signed, int vec, hipStream_t s)
{
    const long long threads = (long long)a.N * a.Ho * a.Wo * (a.C / vec);
    if (threads == 0)
        return hipSuccess;
    long long blocks = (threads + 255) / 256;
    const long long cap = 256LL * 32;
    if (blocks > cap) blocks = cap;
    const dim3 grid((unsigned)blocks);
    const bool mx = a.mode == 1;
    if (is_signed) {
        if (mx) launch_pool_t<true, true>(a, vec, grid, s);
        else launch_pool_t<true, false>(a, vec, grid, s);
    } else {
        if (mx) launch_pool_t<false, true>(a, vec, grid, s);
        else launch_pool_t<false, false>(a, vec, grid, s);
    }
    return hipGetLastError();
}

}  // namespace qnn
