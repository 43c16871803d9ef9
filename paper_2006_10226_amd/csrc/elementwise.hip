// Bandwidth-bound kernels: depthwise conv2d (VALU), standalone requantize
// and qnn.add.
//
// Depthwise (channel multiplier 1) uses the subtract-first form of the
// quantized conv (Sec. III-B, the alternative lowering): each tap
// contributes (x - zp_x) * (w - zp_w[c]) in int32, padded taps contribute
// nothing.  With 9 products per output this is far from any MFMA shape and
// is bound by HBM traffic, so it runs on the vector ALUs.
//
// Requantize is Eq. (5) with the fixed-point multiplier of Sec. III-B; add
// requantizes each operand to the output scale and sums them.
#include "qnn_internal.h"

#include <algorithm>

namespace qnn {

typedef int v4i __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------- depthwise

template <bool VEC4, bool OUT_I32>
__global__ void __launch_bounds__(256) depthwise_kernel(DwArgs a)
{
    const int CV = VEC4 ? 4 : 1;
    const int groups = a.C / CV;
    const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    const long long total = (long long)a.N * a.Ho * a.Wo * groups;
    if (gid >= total)
        return;
    const int g = (int)(gid % groups);
    const int m = (int)(gid / groups);
    const int ow = m % a.Wo, t = m / a.Wo, oh = t % a.Ho, n = t / a.Ho;
    const int c = g * CV;
    int acc[CV];
#pragma unroll
    for (int e = 0; e < CV; ++e)
        acc[e] = 0;
    for (int r = 0; r < a.R; ++r) {
        const int ih = oh * a.sh - a.pt + r * a.dh;
        if ((unsigned)ih >= (unsigned)a.H)
            continue;
        for (int s = 0; s < a.S; ++s) {
            const int iw = ow * a.sw - a.pl + s * a.dw;
            if ((unsigned)iw >= (unsigned)a.W)
                continue;
            const uint8_t *src = a.x + ((size_t)(n * a.H + ih) * a.W + iw) * a.C + c;
            const int32_t *wt = a.wq + (r * a.S + s) * a.C + c;
            if constexpr (VEC4) {
                const uint32_t xv = *(const uint32_t *)src;
                const int4 wv = *(const int4 *)wt;
                const int wk[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t b = (xv >> (8 * e)) & 0xffu;
                    const int xi = a.x_signed ? (int)(int8_t)b : (int)b;
                    acc[e] += (xi - a.zp_x) * wk[e];
                }
            } else {
                const int xi = a.x_signed ? (int)(int8_t)src[0] : (int)src[0];
                acc[0] += (xi - a.zp_x) * wt[0];
            }
        }
    }
    const size_t off = (size_t)m * a.y_ldc + a.y_coff + c;
    if constexpr (OUT_I32) {
        int32_t *yp = (int32_t *)a.y + off;
#pragma unroll
        for (int e = 0; e < CV; ++e)
            yp[e] = (int)((uint32_t)acc[e] + (uint32_t)a.chan[c + e].bconst);
    } else {
        uint8_t *yp = (uint8_t *)a.y + off;
#pragma unroll
        for (int e = 0; e < CV; ++e) {
            const ChanRec cr = a.chan[c + e];
            const int v = (int)((uint32_t)acc[e] + (uint32_t)cr.bconst);
            yp[e] = (uint8_t)clampll(rounding_mul_shift<true>(v, cr.mult, cr.shift, a.rounding) + a.zp_y, a.lo, a.hi);
        }
    }
}

// wq[t][c] = w[t][c] - zp_w[c]; chan[c].bconst = bias[c].
__global__ void __launch_bounds__(256) prep_dw_kernel(const int8_t *w, const int32_t *bias, int RS, int C,
                                                      const int32_t *zpw, int32_t *wq, ChanRec *chan)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= RS * C)
        return;
    const int c = i % C;
    wq[i] = (int)w[i] - zpw[c];
    if (i < C)
        chan[c].bconst = bias ? bias[c] : 0;
}

hipError_t launch_prep_dw(const int8_t *w, const int32_t *bias, int RS, int C, const int32_t *zpw, int32_t *wq,
                          ChanRec *chan, hipStream_t st)
{
    const int n = RS * C;
    hipLaunchKernelGGL(prep_dw_kernel, dim3((n + 255) / 256), dim3(256), 0, st, w, bias, RS, C, zpw, wq, chan);
    return hipGetLastError();
}

hipError_t launch_depthwise(const DwArgs &a, hipStream_t st)
{
    const bool vec = (a.C % 4 == 0) && (a.y_ldc % 4 == 0) && (a.y_coff % 4 == 0) &&
                     (((uintptr_t)a.x & 3) == 0);
    const long long total = (long long)a.N * a.Ho * a.Wo * (vec ? a.C / 4 : a.C);
    dim3 grid((unsigned)((total + 255) / 256)), block(256);
    if (vec) {
        if (a.out_i32) launch_main((depthwise_kernel<true, true>), grid, block, 0, st, a);
        else launch_main((depthwise_kernel<true, false>), grid, block, 0, st, a);
    } else {
        if (a.out_i32) launch_main((depthwise_kernel<false, true>), grid, block, 0, st, a);
        else launch_main((depthwise_kernel<false, false>), grid, block, 0, st, a);
    }
    return hipGetLastError();
}

// ------------------------------------------------------------- elementwise

// dtype codes: 0 uint8, 1 int8, 2 int32
template <int DT>
__device__ __forceinline__ int ld(const void *p, long long i)
{
    if constexpr (DT == 0) return ((const uint8_t *)p)[i];
    else if constexpr (DT == 1) return ((const int8_t *)p)[i];
    else return ((const int32_t *)p)[i];
}

template <int DT>
__device__ __forceinline__ void st(void *p, long long i, int v)
{
    if constexpr (DT == 0) ((uint8_t *)p)[i] = (uint8_t)v;
    else if constexpr (DT == 1) ((int8_t *)p)[i] = (int8_t)v;
    else ((int32_t *)p)[i] = v;
}

// Load 16 consecutive elements starting at a 16-element aligned index.
template <int DT>
__device__ __forceinline__ void ld16(const void *p, long long i0, int v[16])
{
    if constexpr (DT == 2) {
        const int4 *q = (const int4 *)((const int32_t *)p + i0);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int4 u = q[k];
            v[4 * k] = u.x; v[4 * k + 1] = u.y; v[4 * k + 2] = u.z; v[4 * k + 3] = u.w;
        }
    } else {
        const int4 u = *(const int4 *)((const uint8_t *)p + i0);
        const uint32_t w[4] = {(uint32_t)u.x, (uint32_t)u.y, (uint32_t)u.z, (uint32_t)u.w};
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            const uint32_t b = (w[k >> 2] >> (8 * (k & 3))) & 0xffu;
            v[k] = DT == 1 ? (int)(int8_t)b : (int)b;
        }
    }
}

template <int DT>
__device__ __forceinline__ void st16(void *p, long long i0, const int v[16])
{
    if constexpr (DT == 2) {
        int4 *q = (int4 *)((int32_t *)p + i0);
#pragma unroll
        for (int k = 0; k < 4; ++k)
            __builtin_nontemporal_store(v4i{v[4 * k], v[4 * k + 1], v[4 * k + 2], v[4 * k + 3]}, (v4i *)(q + k));
    } else {
        uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
        for (int k = 0; k < 16; ++k)
            w[k >> 2] |= ((uint32_t)v[k] & 0xffu) << (8 * (k & 3));
        __builtin_nontemporal_store(v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]}, (v4i *)((uint8_t *)p + i0));
    }
}

__device__ __forceinline__ int req_one(const ReqArgs &a, int q, int c)
{
    int mult = a.mult, shift = a.shift, zi = a.zp_in, zo = a.zp_out;
    if (a.tab) {
        const int4 t = *(const int4 *)(a.tab + 4 * c);
        mult = t.x; shift = t.y; zi = t.z; zo = t.w;
    }
    return clampll(rounding_mul_shift<true>(q - zi, mult, shift, a.rounding) + zo, a.lo, a.hi);
}

// Each thread handles groups of 16 elements (vector loads/stores when the
// buffers allow it), grid-stride.
template <int XDT, int YDT, bool VEC>
__global__ void __launch_bounds__(256) requantize_kernel(ReqArgs a)
{
    const long long ngroups = (a.count + 15) / 16;
    const long long stride = (long long)gridDim.x * blockDim.x;
    for (long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x; g < ngroups; g += stride) {
        const long long i0 = g * 16;
        int c = a.tab ? (int)(i0 % a.channels) : 0;
        if (VEC && i0 + 16 <= a.count) {
            int v[16];
            ld16<XDT>(a.x, i0, v);
#pragma unroll
            for (int k = 0; k < 16; ++k) {
                v[k] = req_one(a, v[k], c);
                if (a.tab && ++c == a.channels)
                    c = 0;
            }
            st16<YDT>(a.y, i0, v);
        } else {
            for (long long i = i0; i < i0 + 16 && i < a.count; ++i) {
                st<YDT>(a.y, i, req_one(a, ld<XDT>(a.x, i), c));
                if (a.tab && ++c == a.channels)
                    c = 0;
            }
        }
    }
}

// With a.tab_ok each workgroup first tabulates the two terms for every
// operand byte in LDS (256 threads, one byte each), and an element is then
// clamp(tab[a] + tab[256 + b]).
template <int ADT, int BDT, int YDT, bool VEC>
__global__ void __launch_bounds__(256) add_kernel(AddArgs a)
{
    __shared__ int32_t tab[512];
    if (a.tab_ok) {
        const int b = (int)threadIdx.x;
        tab[b] = (int32_t)add_term_a(a, ADT == 1 ? (int)(int8_t)b : b);
        tab[256 + b] = (int32_t)(add_term_b(a, BDT == 1 ? (int)(int8_t)b : b) + a.zp_y);
        __syncthreads();
    }
    const long long ngroups = (a.count + 15) / 16;
    const long long stride = (long long)gridDim.x * blockDim.x;
    for (long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x; g < ngroups; g += stride) {
        const long long i0 = g * 16;
        if (VEC && i0 + 16 <= a.count) {
            int u[16], v[16];
            ld16<ADT>(a.a, i0, u);
            ld16<BDT>(a.b, i0, v);
            if (a.tab_ok) {
#pragma unroll
                for (int k = 0; k < 16; ++k)
                    u[k] = clamp_i32(tab[u[k] & 0xff] + tab[256 + (v[k] & 0xff)], a.lo, a.hi);
            } else {
#pragma unroll
                for (int k = 0; k < 16; ++k)
                    u[k] = add_one(a, u[k], v[k]);
            }
            st16<YDT>(a.y, i0, u);
        } else {
            for (long long i = i0; i < i0 + 16 && i < a.count; ++i)
                st<YDT>(a.y, i, add_one(a, ld<ADT>(a.a, i), ld<BDT>(a.b, i)));
        }
    }
}

static dim3 ew_grid(long long count)
{
    const long long groups = (count + 15) / 16;
    long long blocks = (groups + 255) / 256;
    const long long cap = 256LL * 32;  // enough resident waves to saturate HBM
    if (blocks > cap) blocks = cap;
    if (blocks < 1) blocks = 1;
    return dim3((unsigned)blocks);
}

template <int XDT, int YDT>
static void req_launch(const ReqArgs &a, bool vec, hipStream_t s)
{
    if (vec) launch_main((requantize_kernel<XDT, YDT, true>), ew_grid(a.count), dim3(256), 0, s, a);
    else launch_main((requantize_kernel<XDT, YDT, false>), ew_grid(a.count), dim3(256), 0, s, a);
}

template <int XDT>
static void req_launch_y(const ReqArgs &a, int ydt, bool vec, hipStream_t s)
{
    if (ydt == 0) req_launch<XDT, 0>(a, vec, s);
    else if (ydt == 1) req_launch<XDT, 1>(a, vec, s);
    else req_launch<XDT, 2>(a, vec, s);
}

hipError_t launch_requantize(const ReqArgs &a, int xdt, int ydt, bool aligned, hipStream_t s)
{
    if (xdt == 0) req_launch_y<0>(a, ydt, aligned, s);
    else if (xdt == 1) req_launch_y<1>(a, ydt, aligned, s);
    else req_launch_y<2>(a, ydt, aligned, s);
    return hipGetLastError();
}

template <int ADT, int BDT, int YDT>
static void add_launch(const AddArgs &a, bool vec, hipStream_t s)
{
    if (vec) launch_main((add_kernel<ADT, BDT, YDT, true>), ew_grid(a.count), dim3(256), 0, s, a);
    else launch_main((add_kernel<ADT, BDT, YDT, false>), ew_grid(a.count), dim3(256), 0, s, a);
}

template <int ADT, int BDT>
static void add_launch_y(const AddArgs &a, int ydt, bool vec, hipStream_t s)
{
    if (ydt == 0) add_launch<ADT, BDT, 0>(a, vec, s);
    else add_launch<ADT, BDT, 1>(a, vec, s);
}

template <int ADT>
static void add_launch_b(const AddArgs &a, int bdt, int ydt, bool vec, hipStream_t s)
{
    if (bdt == 0) add_launch_y<ADT, 0>(a, ydt, vec, s);
    else add_launch_y<ADT, 1>(a, ydt, vec, s);
}

hipError_t launch_add(const AddArgs &a, int adt, int bdt, int ydt, bool aligned, hipStream_t s)
{
    if (adt == 0) add_launch_b<0>(a, bdt, ydt, aligned, s);
    else add_launch_b<1>(a, bdt, ydt, aligned, s);
    return hipGetLastError();
}

// AddArgs::tab of a fused residual add: thread b of 256 writes the term of
// the byte b as the first operand (dtype adt) and, plus zp_y, as the
// second (bdt).  The plan builds it only where every term, and so every
// sum, fits 32 bits.
__global__ void __launch_bounds__(256) add_table_kernel(AddArgs a, int adt, int bdt, int32_t *tab)
{
    const int b = (int)threadIdx.x;
    const int x = adt == 1 ? (int)(int8_t)b : b;
    const int y = bdt == 1 ? (int)(int8_t)b : b;
    tab[b] = (int32_t)add_term_a(a, x);
    tab[256 + b] = (int32_t)(add_term_b(a, y) + a.zp_y);
}

hipError_t launch_add_table(const AddArgs &a, int adt, int bdt, int32_t *tab, hipStream_t st)
{
    hipLaunchKernelGGL(add_table_kernel, dim3(1), dim3(256), 0, st, a, adt, bdt, tab);
    return hipGetLastError();
}

// Reads n16 16-byte words of `buf` (grid-stride) so that the L2s and the
// last-level cache hold clean lines of it; `sink` receives a value only in
// the impossible case of an all-ones sum, which keeps the loads alive.
__global__ void __launch_bounds__(256) cache_sweep_kernel(const uint4 *buf, long long n16, int *sink)
{
    uint32_t acc = 0;
    for (long long i = blockIdx.x * 256LL + threadIdx.x; i < n16; i += (long long)gridDim.x * 256) {
        const uint4 v = buf[i];
        acc += v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0xffffffffu)
        *sink = (int)acc;
}

// Legalisation of uint8 weights at plan creation (Sec. III-C): w' = w - 128
// as int8, i.e. each byte XOR 0x80 (the zero point shifts by the same 128).
__global__ void __launch_bounds__(256) flip_bytes_kernel(const uint8_t *in, uint8_t *out, size_t n)
{
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        out[i] = in[i] ^ 0x80u;
}

hipError_t launch_flip_bytes(const uint8_t *in, uint8_t *out, size_t n, hipStream_t st)
{
    if (n == 0)
        return hipSuccess;
    const size_t blocks = std::min<size_t>((n + 255) / 256, 4096);
    hipLaunchKernelGGL(flip_bytes_kernel, dim3((unsigned)blocks), dim3(256), 0, st, in, out, n);
    return hipGetLastError();
}

hipError_t launch_cache_sweep(const void *buf, size_t bytes, int *sink, hipStream_t st)
{
    hipLaunchKernelGGL(cache_sweep_kernel, dim3(4096), dim3(256), 0, st, (const uint4 *)buf, (long long)(bytes / 16),
                       sink);
    return hipGetLastError();
}

}  // namespace qnn
