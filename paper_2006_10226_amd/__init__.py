"""INT8 quantized conv2d / depthwise conv2d / dense with fused requantize for
AMD MI355X (gfx950): a C-ABI HIP library (``libqnn.so``, header
``include/qnn.h``) and its ctypes binding (``paper_2006_10226_amd.qnn``)."""

from . import qnn  # noqa: F401

__all__ = ["qnn"]
