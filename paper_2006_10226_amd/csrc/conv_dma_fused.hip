// Instantiations of the LDS-direct conv kernel (conv_dma_kernel.h) whose
// epilogue applies a residual qnn.add, in a source of their own so that
// they compile beside the plain ones.
#include "conv_dma_kernel.h"

namespace qnn {

namespace {

template <int T>
hipError_t launch_fused_cfg(const ConvArgs &a, hipStream_t st)
{
    constexpr DmaCfg c = kDmaCfg[T];
    if constexpr (dma_fuse_cfg(T)) {
        const int grid = (a.ntiles + 7) / 8 * 8;
        if (a.flip4)
            launch_main((conv_dma_kernel<c.tc, c.tp, c.wc, c.wp, c.ns, true, c.sh, c.ks, false, true>), dim3(grid),
                        dim3(c.wc * c.wp * 64 * c.ks), 0, st, a);
        else
            launch_main((conv_dma_kernel<c.tc, c.tp, c.wc, c.wp, c.ns, false, c.sh, c.ks, false, true>), dim3(grid),
                        dim3(c.wc * c.wp * 64 * c.ks), 0, st, a);
        return hipGetLastError();
    } else {
        return hipErrorInvalidValue;
    }
}

template <int T>
hipError_t launch_fused_from(const ConvArgs &a, int tile, hipStream_t st)
{
    if constexpr (T < DMA_COUNT) {
        if (tile == T)
            return launch_fused_cfg<T>(a, st);
        return launch_fused_from<T + 1>(a, tile, st);
    } else {
        return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_conv_dma_fused(const ConvArgs &a, int tile, hipStream_t st)
{
    if (!a.res || !a.staged || a.ksplit > 1)
        return hipErrorInvalidValue;
    return launch_fused_from<0>(a, tile, st);
}

}  // namespace qnn
