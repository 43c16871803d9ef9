// LDS-direct implicit-GEMM conv launches (kernel in conv_dma_kernel.h) and
// the plan-time kernels of that family: border-class correction table,
// row-pair weight packing, zero-point padded image copies.
#include "conv_dma_kernel.h"

#include <algorithm>

namespace qnn {

// Padding correction table of the border classes (plan preparation): one
// thread per (class, channel) sums the packed weights of the taps outside
// the image and scales by zp_x.  The result wraps to int32 like every other
// term of the accumulator, which is exact whenever the final sum fits.
__global__ void __launch_bounds__(256) border_corr_kernel(const int8_t *wp, int Kpad, int Jpad, int C4, int S, int RS,
                                                          const uint32_t *rmask, const uint32_t *cmask, int ncls,
                                                          int32_t zpx, int32_t *corr)
{
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= ncls * Kpad)
        return;
    const int cls = idx / Kpad, k = idx - cls * Kpad;
    long long sum = 0;
    for (int t = 0; t < RS; ++t) {
        const int r = t / S, s = t - r * S;
        if (((rmask[cls] >> r) & (cmask[cls] >> s) & 1u) == 0) {
            const int8_t *row = wp + (size_t)k * Jpad + (size_t)t * C4;
            for (int c = 0; c < C4; ++c)
                sum += row[c];
        }
    }
    corr[idx] = (int32_t)(uint32_t)(unsigned long long)(sum * zpx);
}

hipError_t launch_border_corr(const int8_t *wp, int Kpad, int Jpad, int C4, int S, int RS, const uint32_t *rmask,
                              const uint32_t *cmask, int ncls, int32_t zpx, int32_t *corr, hipStream_t st)
{
    const int n = ncls * Kpad;
    hipLaunchKernelGGL(border_corr_kernel, dim3((n + 255) / 256), dim3(256), 0, st, wp, Kpad, Jpad, C4, S, RS, rmask,
                       cmask, ncls, zpx, corr);
    return hipGetLastError();
}

// Row-pair packing of the weights for small channel counts (S * C4 <= 32):
// wp[k][64 s + 32 h + b] = w[k][r][b / C4][b % C4] for filter row r = 2 s + h,
// zero where r >= R, b / C4 >= S or b % C4 >= C.  One thread per byte.
__global__ void __launch_bounds__(256) rowpack_weights_kernel(const int8_t *w, int K, int R, int S, int C, int C4,
                                                              int Kpad, int Jpad, int8_t *wp)
{
    const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= (long long)Kpad * Jpad)
        return;
    const int k = (int)(g / Jpad), j = (int)(g - (long long)k * Jpad);
    const int s = j >> 6, h = (j >> 5) & 1, b = j & 31;
    const int r = 2 * s + h, tap = b / C4, c = b - tap * C4;
    int8_t v = 0;
    if (k < K && r < R && tap < S && c < C)
        v = w[(((size_t)k * R + r) * S + tap) * C + c];
    wp[g] = v;
}

// Zero-point padded copy of the image for the row-pair mode:
// out[n][h][w][c] = x[n][h - pt][w - pl][c] inside, zp elsewhere (also in
// the padded channels c >= C).  One thread per padded pixel (C4 <= 32 bytes,
// written as whole dwords; C4 is a multiple of 4).
__global__ void __launch_bounds__(256) pad_image_kernel(const uint8_t *x, int N, int H, int W, int C, int Hp, int Wp,
                                                        int C4, int pt, int pl, uint8_t zp, uint8_t *out)
{
    // block (bx, by): padded pixels 256 bx .. of the rows by, by + gridDim.y,
    // ...; the row split is uniform over the block (scalar arithmetic)
    const int w = (int)(blockIdx.x * blockDim.x + threadIdx.x);
    if (w >= Wp)
        return;
    const int iw = w - pl;
    const bool col_in = (unsigned)iw < (unsigned)W;
    for (int row = (int)blockIdx.y; row < N * Hp; row += (int)gridDim.y) {
        const int n = row / Hp, h = row - n * Hp;
        const int ih = h - pt;
        const bool in = col_in && (unsigned)ih < (unsigned)H;
        const uint8_t *src = x + ((size_t)(n * H + (in ? ih : 0)) * W + (in ? iw : 0)) * C;
        uint32_t *dst = (uint32_t *)(out + ((size_t)row * Wp + w) * C4);
        for (int c0 = 0; c0 < C4; c0 += 4) {
            uint32_t v = 0;
            for (int e = 0; e < 4; ++e) {
                const int c = c0 + e;
                const uint32_t b = (in && c < C) ? src[c] : zp;
                v |= b << (8 * e);
            }
            dst[c0 >> 2] = v;
        }
    }
}

// The same copy for 3-channel images with W % 4 == 0 and a 4-byte aligned
// x: one wave per padded row (four rows per block); lane t < W / 4 turns
// source pixels 4t .. 4t + 3 (three aligned dwords) into four padded
// pixels (the fourth byte zp), the lanes after them fill the pad columns,
// and rows outside the image are filled whole.
__global__ void __launch_bounds__(256) pad_rgb_kernel(const uint8_t *x, int N, int H, int W, int Hp, int Wp, int pt,
                                                      int pl, uint8_t zp, uint8_t *out)
{
    const int row = (int)blockIdx.x * 4 + (int)(threadIdx.x >> 6);   // n * Hp + h
    if (row >= N * Hp)
        return;
    const int lane = (int)(threadIdx.x & 63);
    const int n = row / Hp, h = row - n * Hp;
    const int ih = h - pt;
    const bool row_in = (unsigned)ih < (unsigned)H;
    const uint32_t fill = 0x01010101u * zp, top = (uint32_t)zp << 24;
    uint32_t *dst = (uint32_t *)(out + (size_t)row * Wp * 4);
    const int groups = W >> 2;
    for (int t = lane; t < groups + (Wp - W); t += 64) {
        if (t < groups) {
            uint32_t o0 = fill, o1 = fill, o2 = fill, o3 = fill;
            if (row_in) {
                const uint32_t *src = (const uint32_t *)(x + ((size_t)(n * H + ih) * W + 4 * t) * 3);
                const uint32_t d0 = src[0], d1 = src[1], d2 = src[2];
                o0 = (d0 & 0xffffffu) | top;
                o1 = (((d0 >> 24) | (d1 << 8)) & 0xffffffu) | top;
                o2 = (((d1 >> 16) | (d2 << 16)) & 0xffffffu) | top;
                o3 = (d2 >> 8) | top;
            }
            uint32_t *p = dst + pl + 4 * t;
            p[0] = o0;
            p[1] = o1;
            p[2] = o2;
            p[3] = o3;
        } else {
            const int q = t - groups;        // pad column: the pl left ones, then the right ones
            dst[q < pl ? q : W + q] = fill;
        }
    }
}

hipError_t launch_rowpack_weights(const int8_t *w, int K, int R, int S, int C, int C4, int Kpad, int Jpad, int8_t *wp,
                                  hipStream_t st)
{
    const long long n = (long long)Kpad * Jpad;
    hipLaunchKernelGGL(rowpack_weights_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, w, K, R, S, C, C4,
                       Kpad, Jpad, wp);
    return hipGetLastError();
}

hipError_t launch_pad_image(const uint8_t *x, int N, int H, int W, int C, int Hp, int Wp, int C4, int pt, int pl,
                            uint8_t zp, uint8_t *out, hipStream_t st)
{
    const long long rows = (long long)N * Hp;
    if (rows * Wp == 0)
        return hipSuccess;
    if (rows >= (1LL << 31))
        return hipErrorInvalidValue;
    if (C == 3 && C4 == 4 && W % 4 == 0 && ((uintptr_t)x & 3) == 0 && pl >= 0 && Wp >= W + pl) {
        hipLaunchKernelGGL(pad_rgb_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, x, N, H, W, Hp, Wp, pt,
                           pl, zp, out);
        return hipGetLastError();
    }
    const dim3 grid((unsigned)((Wp + 255) / 256), (unsigned)std::min<long long>(rows, 65535));
    hipLaunchKernelGGL(pad_image_kernel, grid, dim3(256), 0, st, x, N, H, W, C, Hp, Wp, C4, pt, pl, zp, out);
    return hipGetLastError();
}

// DmaTile -> tile, wave grid, stage count, short-reduction form, K-step
// groups.

TileShape dma_tile_shape(int tile)
{
    return {kDmaCfg[tile].tc, kDmaCfg[tile].tp, 64};
}

// ring configurations with a split-reduction instantiation
static constexpr bool dma_split_cfg(int t)
{
    return t == DMA_128x128_S4 || t == DMA_128x128_S8 || t == DMA_128x64_S4 || t == DMA_64x128_S4 ||
           t == DMA_64x64_S4 || t == DMA_64x64_S8 || t == DMA_256x128_S4 || t == DMA_128x256_S4 ||
           t == DMA_256x128_W4 || t == DMA_128x256_W4;
}

bool dma_splits(int tile)
{
    return tile >= 0 && tile < DMA_COUNT && dma_split_cfg(tile);
}

int dma_wave_tile(int tile)
{
    return kDmaCfg[tile].tc / kDmaCfg[tile].wc * (kDmaCfg[tile].tp / kDmaCfg[tile].wp);
}

int dma_threads(int tile)
{
    return kDmaCfg[tile].wc * kDmaCfg[tile].wp * 64 * kDmaCfg[tile].ks;
}

int dma_split(int tile)
{
    return kDmaCfg[tile].ks;
}

int dma_stages(int tile)
{
    return kDmaCfg[tile].ns;
}

bool dma_short(int tile)
{
    return kDmaCfg[tile].sh;
}

template <int T>
static hipError_t launch_dma_cfg(const ConvArgs &a, hipStream_t st)
{
    constexpr DmaCfg c = kDmaCfg[T];
    const int grid = (a.ntiles + 7) / 8 * 8;
    if (c.sh && a.nk > c.ns)
        return hipErrorInvalidValue;   // more K-steps than the short form holds
    if (c.ks > 1 && a.rowpack)
        return hipErrorInvalidValue;   // the row-pair walk steps one K-step at a time
    if (a.res)
        return a.ksplit > 1 ? hipErrorInvalidValue : launch_conv_dma_fused(a, T, st);
    if (a.ksplit > 1) {
        if constexpr (dma_split_cfg(T)) {
            if (a.rowpack || a.C % 64 != 0 || !a.part || !a.cnt)
                return hipErrorInvalidValue;   // split parts start at whole 64-channel steps
            const int units = (a.ntiles * a.ksplit + 7) / 8 * 8;
            if (a.flip4)
                launch_main((conv_dma_kernel<c.tc, c.tp, c.wc, c.wp, c.ns, true, false, 1, true>),
                                   dim3(units), dim3(c.wc * c.wp * 64), 0, st, a);
            else
                launch_main((conv_dma_kernel<c.tc, c.tp, c.wc, c.wp, c.ns, false, false, 1, true>),
                                   dim3(units), dim3(c.wc * c.wp * 64), 0, st, a);
            return hipGetLastError();
        } else {
            return hipErrorInvalidValue;
        }
    }
    if (a.flip4)
        launch_main((conv_dma_kernel<c.tc, c.tp, c.wc, c.wp, c.ns, true, c.sh, c.ks>), dim3(grid),
                           dim3(c.wc * c.wp * 64 * c.ks), 0, st, a);
    else
        launch_main((conv_dma_kernel<c.tc, c.tp, c.wc, c.wp, c.ns, false, c.sh, c.ks>), dim3(grid),
                           dim3(c.wc * c.wp * 64 * c.ks), 0, st, a);
    return hipGetLastError();
}

template <int T>
static hipError_t launch_dma_from(const ConvArgs &a, int tile, hipStream_t st)
{
    if constexpr (T < DMA_COUNT) {
        if (tile == T)
            return launch_dma_cfg<T>(a, st);
        return launch_dma_from<T + 1>(a, tile, st);
    } else {
        return hipErrorInvalidValue;
    }
}

hipError_t launch_conv_dma(const ConvArgs &a, int tile, hipStream_t st)
{
    return launch_dma_from<0>(a, tile, st);
}

}  // namespace qnn
