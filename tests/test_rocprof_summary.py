"""Kernel symbols as rocprofv3 prints them map to bench.py's kernel-group
names (the profile summaries join the two by these names)."""
from paper_2006_10226_amd.rocprof_summary import group_of


def test_template_symbols():
    cases = {
        "void qnn::conv_tap_kernel<128, 64, 128, 4, 1, false>(qnn::ConvArgs)":
            "conv_tap tile=128x64x128 threads=256 stages=2",
        "void qnn::conv_tap_kernel<128, 64, 128, 4, 1, true>(qnn::ConvArgs)":
            "conv_tap tile=128x64x128 threads=256 stages=2 +add",
        "void qnn::conv_dma_kernel<64, 128, 2, 2, 1, true, true, 1, false, false>(qnn::ConvArgs)":
            "conv_dma tile=64x128x64 threads=256 stages=1s",
        "void qnn::conv_dma_kernel<128, 64, 2, 2, 8, false, false, 2, false, false>(qnn::ConvArgs)":
            "conv_dma tile=128x64x64 threads=512 stages=8",
        "void qnn::conv_dma_kernel<128, 128, 2, 2, 4, true, false, 1, true, false>(qnn::ConvArgs)":
            "conv_dma tile=128x128x64 threads=256 stages=4 ksplit",
        "void qnn::conv_dma_kernel<64, 128, 2, 2, 1, false, true, 1, false, true>(qnn::ConvArgs)":
            "conv_dma tile=64x128x64 threads=256 stages=1s +add",
        "void qnn::depthwise3_band_kernel<8, 2, true, false, 1>(qnn::DwArgs)": "depthwise",
        "void qnn::add_kernel<1, 1, 1, true>(qnn::AddArgs)": "add",
    }
    for sym, group in cases.items():
        assert group_of(sym) == group, sym
