"""Python binding of libqnn (ctypes): argument marshalling only.

Every computation runs in the HIP kernels of ``libqnn.so``; PyTorch supplies
device memory and the current stream.  The library must have been built
(``python -m paper_2006_10226_amd.build`` or ``__graft_entry__.build()``);
the first call into it raises ImportError when it is missing -- there is no
CPU fallback.

Conventions follow include/qnn.h: activations NHWC, conv weights OHWI,
depthwise weights [R][S][C], dense weights [N][K]; scales and zero points are
Python numbers or sequences (per tensor or per output channel).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple, Union

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libqnn.so")

UINT8, INT8, INT32 = 0, 1, 2
HALF_UP, HALF_AWAY, TWO_STAGE = 0, 1, 2
_TORCH_DT = {torch.uint8: UINT8, torch.int8: INT8, torch.int32: INT32}
_NAME_DT = {"u8": UINT8, "i8": INT8, "i32": INT32}
_DT_TORCH = {UINT8: torch.uint8, INT8: torch.int8, INT32: torch.int32}
_ROUND = {"half_up": HALF_UP, "half_away": HALF_AWAY, "two_stage": TWO_STAGE}
INT32_MIN, INT32_MAX = -(2**31), 2**31 - 1

STATUS = ["QNN_OK", "QNN_ERR_NULL", "QNN_ERR_SHAPE", "QNN_ERR_DTYPE", "QNN_ERR_QPARAM",
          "QNN_ERR_OVERFLOW", "QNN_ERR_UNSUPPORTED", "QNN_ERR_HIP", "QNN_ERR_ALLOC"]

# Every symbol the public header declares.
EXPORTS = [
    "qnn_abi_version", "qnn_last_error", "qnn_status_string", "qnn_quantize_multiplier",
    "qnn_conv2d", "qnn_depthwise_conv2d", "qnn_dense", "qnn_requantize", "qnn_add",
    "qnn_pool2d",
    "qnn_conv2d_plan_create", "qnn_depthwise_conv2d_plan_create", "qnn_dense_plan_create",
    "qnn_conv2d_plan_create_wt", "qnn_depthwise_conv2d_plan_create_wt", "qnn_dense_plan_create_wt",
    "qnn_requantize_plan_create", "qnn_plan_run", "qnn_plan_run_timed", "qnn_time_next_kernel", "qnn_plan_run_noalloc",
    "qnn_plan_set_residual", "qnn_plan_run_residual", "qnn_plan_workspace_size",
    "qnn_plan_describe", "qnn_set_tuning_file", "qnn_plan_destroy",
]


class QnnError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        self.status_name = STATUS[status] if 0 <= status < len(STATUS) else f"status {status}"
        super().__init__(f"{self.status_name}: {message}")


class QParams(ctypes.Structure):
    _fields_ = [("scale", ctypes.POINTER(ctypes.c_float)),
                ("zero_point", ctypes.POINTER(ctypes.c_int32)),
                ("n", ctypes.c_int32)]


class ConvParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("stride_h", "stride_w", "pad_top", "pad_left", "pad_bottom", "pad_right", "dil_h", "dil_w")]


class Clamp(ctypes.Structure):
    _fields_ = [("lo", ctypes.c_int32), ("hi", ctypes.c_int32)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libqnn.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it first (python -m paper_2006_10226_amd.build)")
    L = ctypes.CDLL(LIB_PATH)
    P, i32, i64, st = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_int
    L.qnn_abi_version.restype = i32
    L.qnn_last_error.restype = ctypes.c_char_p
    L.qnn_status_string.restype = ctypes.c_char_p
    L.qnn_status_string.argtypes = [st]
    L.qnn_quantize_multiplier.argtypes = [ctypes.c_double, P, P]
    L.qnn_quantize_multiplier.restype = st
    conv_args = [P, st, i32, i32, i32, i32, QParams, P, i32, i32, i32, QParams, P, ConvParams,
                 P, st, QParams, Clamp, st, i32, i32]
    L.qnn_conv2d.argtypes = [P] + conv_args
    L.qnn_conv2d.restype = st
    dw_args = [P, st, i32, i32, i32, i32, QParams, P, i32, i32, QParams, P, ConvParams,
               P, st, QParams, Clamp, st, i32, i32]
    L.qnn_depthwise_conv2d.argtypes = [P] + dw_args
    L.qnn_depthwise_conv2d.restype = st
    L.qnn_dense.argtypes = [P, P, st, i32, i32, QParams, P, i32, QParams, P, P, st, QParams, Clamp, st, i32]
    L.qnn_dense.restype = st
    L.qnn_requantize.argtypes = [P, P, st, i64, i32, QParams, P, st, QParams, Clamp, st]
    L.qnn_requantize.restype = st
    L.qnn_add.argtypes = [P, P, st, QParams, P, st, QParams, i64, P, st, QParams, Clamp, st]
    L.qnn_add.restype = st
    L.qnn_pool2d.argtypes = [P, P, st, i32, i32, i32, i32, i32, i32, ConvParams, st, i32, i32, P, st]
    L.qnn_pool2d.restype = st
    PP = ctypes.POINTER(ctypes.c_void_p)
    L.qnn_conv2d_plan_create.argtypes = [PP, P, st, i32, i32, i32, i32, QParams, P, i32, i32, i32,
                                         QParams, P, ConvParams, st, QParams, Clamp, st, i32, i32]
    L.qnn_conv2d_plan_create.restype = st
    L.qnn_depthwise_conv2d_plan_create.argtypes = [PP, P, st, i32, i32, i32, i32, QParams, P, i32, i32,
                                                   QParams, P, ConvParams, st, QParams, Clamp, st, i32, i32]
    L.qnn_depthwise_conv2d_plan_create.restype = st
    L.qnn_dense_plan_create.argtypes = [PP, P, st, i32, i32, QParams, P, i32, QParams, P, st, QParams,
                                        Clamp, st, i32]
    L.qnn_dense_plan_create.restype = st
    L.qnn_conv2d_plan_create_wt.argtypes = [PP, P, st, i32, i32, i32, i32, QParams, P, st, i32, i32, i32,
                                            QParams, P, ConvParams, st, QParams, Clamp, st, i32, i32]
    L.qnn_conv2d_plan_create_wt.restype = st
    L.qnn_depthwise_conv2d_plan_create_wt.argtypes = [PP, P, st, i32, i32, i32, i32, QParams, P, st, i32, i32,
                                                      QParams, P, ConvParams, st, QParams, Clamp, st, i32, i32]
    L.qnn_depthwise_conv2d_plan_create_wt.restype = st
    L.qnn_dense_plan_create_wt.argtypes = [PP, P, st, i32, i32, QParams, P, st, i32, QParams, P, st, QParams,
                                           Clamp, st, i32]
    L.qnn_dense_plan_create_wt.restype = st
    L.qnn_requantize_plan_create.argtypes = [PP, P, st, i64, i32, QParams, st, QParams, Clamp, st]
    L.qnn_requantize_plan_create.restype = st
    L.qnn_plan_run.argtypes = [P, P, P, P, P]
    L.qnn_plan_run.restype = st
    L.qnn_plan_run_timed.argtypes = [P, P, P, P, P, P, P]
    L.qnn_plan_run_timed.restype = st
    L.qnn_time_next_kernel.argtypes = [P, P]
    L.qnn_time_next_kernel.restype = st
    L.qnn_plan_run_noalloc.argtypes = [P, P, P, P]
    L.qnn_plan_run_noalloc.restype = st
    L.qnn_plan_set_residual.argtypes = [P, st, QParams, i32, i32, st, QParams, Clamp, st]
    L.qnn_plan_set_residual.restype = st
    L.qnn_plan_run_residual.argtypes = [P, P, P, P, P, P]
    L.qnn_plan_run_residual.restype = st
    L.qnn_plan_workspace_size.argtypes = [P]
    L.qnn_plan_workspace_size.restype = ctypes.c_size_t
    L.qnn_plan_describe.argtypes = [P]
    L.qnn_plan_describe.restype = ctypes.c_char_p
    L.qnn_set_tuning_file.argtypes = [ctypes.c_char_p]
    L.qnn_set_tuning_file.restype = st
    L.qnn_plan_destroy.argtypes = [P]
    L.qnn_plan_destroy.restype = None
    _lib = L
    return L


def _check(status: int):
    if status != 0:
        raise QnnError(status, lib().qnn_last_error().decode())


class _Q:
    """Host arrays behind a qnn_qparams (kept alive for the call)."""

    def __init__(self, scale, zp, n: Optional[int] = None):
        s = np.atleast_1d(np.asarray(scale, dtype=np.float32))
        z = np.atleast_1d(np.asarray(zp, dtype=np.int32))
        if n is None:
            n = max(s.size, z.size)
        if s.size == 1 and n > 1:
            s = np.full(n, s[0], np.float32)
        if z.size == 1 and n > 1:
            z = np.full(n, z[0], np.int32)
        self.s = np.ascontiguousarray(s)
        self.z = np.ascontiguousarray(z)
        self.q = QParams(self.s.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                         self.z.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), int(n))


def _per_tensor_or_channel(scale, zp):
    s = np.atleast_1d(np.asarray(scale, dtype=np.float32))
    z = np.atleast_1d(np.asarray(zp, dtype=np.int32))
    return _Q(s, z, max(s.size, z.size))


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dt(t: torch.Tensor) -> int:
    if t.dtype not in _TORCH_DT:
        raise TypeError(f"unsupported dtype {t.dtype}")
    return _TORCH_DT[t.dtype]


def _clamp(act: Optional[Tuple[int, int]]) -> Clamp:
    if act is None:
        return Clamp(INT32_MIN, INT32_MAX)
    return Clamp(int(max(INT32_MIN, act[0])), int(min(INT32_MAX, act[1])))


def _cp(stride, pads, dil) -> ConvParams:
    sh, sw = (stride, stride) if isinstance(stride, int) else stride
    dh, dw = (dil, dil) if isinstance(dil, int) else dil
    pt, pl, pb, pr = (pads,) * 4 if isinstance(pads, int) else pads
    return ConvParams(sh, sw, pt, pl, pb, pr, dh, dw)


def out_hw(H, W, R, S, stride=1, pads=0, dil=1):
    cp = _cp(stride, pads, dil)
    Ho = (H + cp.pad_top + cp.pad_bottom - cp.dil_h * (R - 1) - 1) // cp.stride_h + 1
    Wo = (W + cp.pad_left + cp.pad_right - cp.dil_w * (S - 1) - 1) // cp.stride_w + 1
    return Ho, Wo


def _contig(t: torch.Tensor, name: str):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _check_out(out: torch.Tensor, lead, ydt, whole=False):
    shape = tuple(out.shape) if whole else tuple(out.shape[:-1])
    if shape != tuple(lead) or out.dtype != _DT_TORCH[ydt]:
        raise ValueError(f"out is {tuple(out.shape)} {out.dtype}; expected leading dims {tuple(lead)} "
                         f"and dtype {_DT_TORCH[ydt]}")


def quantize_multiplier(M: float) -> Tuple[int, int]:
    m, s = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().qnn_quantize_multiplier(float(M), ctypes.byref(m), ctypes.byref(s)))
    return m.value, s.value


def time_next_kernel(start, stop):
    """The next main kernel launched from this thread records the two
    torch.cuda.Event objects at its own start and end."""
    for e in (start, stop):
        if not e.cuda_event:   # torch creates its events on first record
            e.record()
    _check(lib().qnn_time_next_kernel(ctypes.c_void_p(start.cuda_event), ctypes.c_void_p(stop.cuda_event)))


def set_tuning_file(path: Optional[str]):
    """Read kernel choices from, and append timed ones to, a text file
    (None: stop); see qnn_set_tuning_file."""
    _check(lib().qnn_set_tuning_file(None if path is None else os.fsencode(path)))


def abi_version() -> int:
    return lib().qnn_abi_version()


# ---------------------------------------------------------------- plans

class Plan:
    """A prepared conv / depthwise / dense / requantize (owns device memory)."""

    def __init__(self, handle: ctypes.c_void_p, in_shape, in_dtype, out_shape, out_dtype, y_ldc_shape=None):
        self._h = handle
        self.in_shape = tuple(in_shape)
        self.in_dtype = in_dtype
        self.out_shape = tuple(out_shape)
        self.out_dtype = out_dtype
        self.y_ldc_shape = tuple(y_ldc_shape or out_shape)

    @property
    def handle(self):
        return self._h

    @property
    def workspace_size(self) -> int:
        return int(lib().qnn_plan_workspace_size(self._h))

    def describe(self) -> str:
        return lib().qnn_plan_describe(self._h).decode()

    def set_residual(self, r_dtype, r_scale, r_zp, o_scale, o_zp, o_dtype="u8", act=None, rounding="half_up",
                     r_ldc=None, r_coff=0):
        """qnn_plan_set_residual: the plan then stores qnn.add(its conv
        output, a residual of the output's pixels) with the output qparams
        o_*; run it with run(x, out, workspace, residual=r), r of shape
        (N, Ho, Wo, r_ldc) (r_ldc defaults to the output channels)."""
        N, Ho, Wo, K = self.out_shape
        r_ldc = K if r_ldc is None else r_ldc
        rdt, odt = _NAME_DT[r_dtype], _NAME_DT[o_dtype]
        rq, oq = _Q(r_scale, r_zp, 1), _Q(o_scale, o_zp, 1)
        _check(lib().qnn_plan_set_residual(self._h, rdt, rq.q, r_ldc, r_coff, odt, oq.q, _clamp(act),
                                           _ROUND[rounding]))
        self.out_dtype = _DT_TORCH[odt]
        self.residual = ((N, Ho, Wo, r_ldc), _DT_TORCH[rdt])
        return self

    def new_output(self, device="cuda"):
        return torch.empty(self.y_ldc_shape or self.out_shape, dtype=self.out_dtype, device=device)

    def run(self, x: torch.Tensor, out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
            stream=None, residual: Optional[torch.Tensor] = None) -> torch.Tensor:
        """Run on x (shape and dtype fixed at creation); the kernels trust the
        sizes, so they are checked here.  A plan with a fused add
        (set_residual) takes its residual tensor."""
        _contig(x, "x")
        if tuple(x.shape) != self.in_shape or x.dtype != self.in_dtype:
            raise ValueError(f"x is {tuple(x.shape)} {x.dtype}, the plan expects {self.in_shape} {self.in_dtype}")
        if out is None:
            out = self.new_output(x.device)
        _contig(out, "out")
        if tuple(out.shape) != self.y_ldc_shape or out.dtype != self.out_dtype:
            raise ValueError(f"out is {tuple(out.shape)} {out.dtype}, the plan writes {self.y_ldc_shape} "
                             f"{self.out_dtype}")
        if self.workspace_size and workspace is not None and workspace.numel() * workspace.element_size() < \
                self.workspace_size:
            raise ValueError("workspace is smaller than the plan needs")
        fused = getattr(self, "residual", None)
        if (fused is None) != (residual is None):
            raise ValueError("a residual goes with a plan that has a fused add (set_residual), and only with one")
        if fused is not None:
            _contig(residual, "residual")
            if tuple(residual.shape) != fused[0] or residual.dtype != fused[1]:
                raise ValueError(f"residual is {tuple(residual.shape)} {residual.dtype}, the plan expects "
                                 f"{fused[0]} {fused[1]}")
            _check(lib().qnn_plan_run_residual(self._h, _stream(stream), _ptr(x), _ptr(residual), _ptr(out),
                                               _ptr(workspace)))
            return out
        _check(lib().qnn_plan_run(self._h, _stream(stream), _ptr(x), _ptr(out), _ptr(workspace)))
        return out

    def run_timed(self, x: torch.Tensor, out: torch.Tensor, workspace, start, stop, stream=None):
        """qnn_plan_run_timed: start / stop (torch.cuda.Event with timing)
        are recorded at the main kernel's own start and end."""
        for e in (start, stop):
            if not e.cuda_event:   # torch creates its events on first record
                e.record()
        _check(lib().qnn_plan_run_timed(self._h, _stream(stream), _ptr(x), _ptr(out), _ptr(workspace),
                                        ctypes.c_void_p(start.cuda_event), ctypes.c_void_p(stop.cuda_event)))
        return out

    def run_noalloc(self, x: torch.Tensor, out: torch.Tensor, stream=None) -> torch.Tensor:
        """qnn_plan_run_noalloc: the workspace is the library's static device
        array; out must be given (nothing is allocated)."""
        _contig(x, "x")
        _contig(out, "out")
        if tuple(x.shape) != self.in_shape or x.dtype != self.in_dtype:
            raise ValueError(f"x is {tuple(x.shape)} {x.dtype}, the plan expects {self.in_shape} {self.in_dtype}")
        if tuple(out.shape) != self.y_ldc_shape or out.dtype != self.out_dtype:
            raise ValueError(f"out is {tuple(out.shape)} {out.dtype}, the plan writes {self.y_ldc_shape} "
                             f"{self.out_dtype}")
        _check(lib().qnn_plan_run_noalloc(self._h, _stream(stream), _ptr(x), _ptr(out)))
        return out

    def close(self):
        if self._h:
            lib().qnn_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def conv2d_plan(x_shape, x_dtype, x_scale, x_zp, w: torch.Tensor, w_scale, w_zp, bias=None,
                stride=1, pads=0, dil=1, y_scale=1.0, y_zp=0, y_dtype="u8", act=None,
                rounding="half_up", y_ldc=None, y_coff=0, stream=None) -> Plan:
    N, H, W, C = x_shape
    _contig(w, "w")
    K, R, S, Cw = w.shape
    if Cw != C:
        raise ValueError("weight Cin does not match x")
    cp = _cp(stride, pads, dil)
    Ho, Wo = out_hw(H, W, R, S, stride, pads, dil)
    y_ldc = K if y_ldc is None else y_ldc
    xq, wq, yq = _Q(x_scale, x_zp, 1), _per_tensor_or_channel(w_scale, w_zp), _Q(y_scale, y_zp, 1)
    h = ctypes.c_void_p()
    if w.dtype == torch.uint8:   # asymmetric uint8 weights, legalised at creation
        _check(lib().qnn_conv2d_plan_create_wt(ctypes.byref(h), _stream(stream), _NAME_DT[x_dtype], N, H, W, C,
                                               xq.q, _ptr(w), UINT8, K, R, S, wq.q, _ptr(bias), cp,
                                               _NAME_DT[y_dtype], yq.q, _clamp(act), _ROUND[rounding], y_ldc,
                                               y_coff))
    else:
        _check(lib().qnn_conv2d_plan_create(ctypes.byref(h), _stream(stream), _NAME_DT[x_dtype], N, H, W, C, xq.q,
                                            _ptr(w), K, R, S, wq.q, _ptr(bias), cp, _NAME_DT[y_dtype], yq.q,
                                            _clamp(act), _ROUND[rounding], y_ldc, y_coff))
    return Plan(h, x_shape, _DT_TORCH[_NAME_DT[x_dtype]], (N, Ho, Wo, K), _DT_TORCH[_NAME_DT[y_dtype]],
                (N, Ho, Wo, y_ldc))


def depthwise_conv2d_plan(x_shape, x_dtype, x_scale, x_zp, w: torch.Tensor, w_scale, w_zp, bias=None,
                          stride=1, pads=0, dil=1, y_scale=1.0, y_zp=0, y_dtype="u8", act=None,
                          rounding="half_up", y_ldc=None, y_coff=0, stream=None) -> Plan:
    N, H, W, C = x_shape
    _contig(w, "w")
    R, S, Cw = w.shape
    if Cw != C:
        raise ValueError("depthwise weight channels do not match x")
    cp = _cp(stride, pads, dil)
    Ho, Wo = out_hw(H, W, R, S, stride, pads, dil)
    y_ldc = C if y_ldc is None else y_ldc
    xq, wq, yq = _Q(x_scale, x_zp, 1), _per_tensor_or_channel(w_scale, w_zp), _Q(y_scale, y_zp, 1)
    h = ctypes.c_void_p()
    if w.dtype == torch.uint8:
        _check(lib().qnn_depthwise_conv2d_plan_create_wt(ctypes.byref(h), _stream(stream), _NAME_DT[x_dtype], N, H,
                                                         W, C, xq.q, _ptr(w), UINT8, R, S, wq.q, _ptr(bias), cp,
                                                         _NAME_DT[y_dtype], yq.q, _clamp(act), _ROUND[rounding],
                                                         y_ldc, y_coff))
    else:
        _check(lib().qnn_depthwise_conv2d_plan_create(ctypes.byref(h), _stream(stream), _NAME_DT[x_dtype], N, H, W,
                                                      C, xq.q, _ptr(w), R, S, wq.q, _ptr(bias), cp,
                                                      _NAME_DT[y_dtype], yq.q, _clamp(act), _ROUND[rounding],
                                                      y_ldc, y_coff))
    return Plan(h, x_shape, _DT_TORCH[_NAME_DT[x_dtype]], (N, Ho, Wo, C), _DT_TORCH[_NAME_DT[y_dtype]],
                (N, Ho, Wo, y_ldc))


def dense_plan(M, K, x_dtype, x_scale, x_zp, w: torch.Tensor, w_scale, w_zp, bias=None, y_scale=1.0, y_zp=0,
               y_dtype="i8", act=None, rounding="half_up", y_ldc=None, stream=None) -> Plan:
    _contig(w, "w")
    Nd, Kw = w.shape
    if Kw != K:
        raise ValueError("dense weight K does not match x")
    y_ldc = Nd if y_ldc is None else y_ldc
    xq, wq, yq = _Q(x_scale, x_zp, 1), _per_tensor_or_channel(w_scale, w_zp), _Q(y_scale, y_zp, 1)
    h = ctypes.c_void_p()
    if w.dtype == torch.uint8:
        _check(lib().qnn_dense_plan_create_wt(ctypes.byref(h), _stream(stream), _NAME_DT[x_dtype], M, K, xq.q,
                                              _ptr(w), UINT8, Nd, wq.q, _ptr(bias), _NAME_DT[y_dtype], yq.q,
                                              _clamp(act), _ROUND[rounding], y_ldc))
    else:
        _check(lib().qnn_dense_plan_create(ctypes.byref(h), _stream(stream), _NAME_DT[x_dtype], M, K, xq.q, _ptr(w),
                                           Nd, wq.q, _ptr(bias), _NAME_DT[y_dtype], yq.q, _clamp(act),
                                           _ROUND[rounding], y_ldc))
    return Plan(h, (M, K), _DT_TORCH[_NAME_DT[x_dtype]], (M, Nd), _DT_TORCH[_NAME_DT[y_dtype]], (M, y_ldc))


def requantize_plan(shape, x_dtype, x_scale, x_zp, y_scale, y_zp, y_dtype="u8", act=None,
                    rounding="half_up", stream=None) -> Plan:
    channels = shape[-1] if len(shape) else 1
    count = int(np.prod(shape)) if len(shape) else 1
    xq, yq = _per_tensor_or_channel(x_scale, x_zp), _per_tensor_or_channel(y_scale, y_zp)
    h = ctypes.c_void_p()
    _check(lib().qnn_requantize_plan_create(ctypes.byref(h), _stream(stream), _NAME_DT[x_dtype], count, channels,
                                            xq.q, _NAME_DT[y_dtype], yq.q, _clamp(act), _ROUND[rounding]))
    return Plan(h, shape, _DT_TORCH[_NAME_DT[x_dtype]], shape, _DT_TORCH[_NAME_DT[y_dtype]])


# ---------------------------------------------------------------- one-shot ops

def conv2d(x: torch.Tensor, x_scale, x_zp, w: torch.Tensor, w_scale, w_zp, bias=None, stride=1, pads=0,
           dil=1, y_scale=1.0, y_zp=0, y_dtype="u8", act=None, rounding="half_up",
           out: Optional[torch.Tensor] = None, y_coff=0, stream=None) -> torch.Tensor:
    """qnn.conv2d + bias + requantize + clamp; NHWC x, OHWI w (device tensors).

    With ``out`` given (NHWC, last dim = row stride), the result is written to
    channels [y_coff, y_coff + K) of it (a concat slice)."""
    _contig(x, "x")
    _contig(w, "w")
    N, H, W, C = x.shape
    K, R, S, _ = w.shape
    Ho, Wo = out_hw(H, W, R, S, stride, pads, dil)
    ydt = _NAME_DT[y_dtype]
    if out is None:
        out = torch.empty((N, Ho, Wo, K), dtype=_DT_TORCH[ydt], device=x.device)
    _contig(out, "out")
    _check_out(out, (N, Ho, Wo), ydt)
    xq, wq, yq = _Q(x_scale, x_zp, 1), _per_tensor_or_channel(w_scale, w_zp), _Q(y_scale, y_zp, 1)
    _check(lib().qnn_conv2d(_stream(stream), _ptr(x), _dt(x), N, H, W, C, xq.q, _ptr(w), K, R, S, wq.q,
                            _ptr(bias), _cp(stride, pads, dil), _ptr(out), ydt, yq.q, _clamp(act),
                            _ROUND[rounding], out.shape[-1], y_coff))
    return out


def depthwise_conv2d(x: torch.Tensor, x_scale, x_zp, w: torch.Tensor, w_scale, w_zp, bias=None, stride=1,
                     pads=0, dil=1, y_scale=1.0, y_zp=0, y_dtype="u8", act=None, rounding="half_up",
                     out: Optional[torch.Tensor] = None, y_coff=0, stream=None) -> torch.Tensor:
    _contig(x, "x")
    _contig(w, "w")
    N, H, W, C = x.shape
    R, S, _ = w.shape
    Ho, Wo = out_hw(H, W, R, S, stride, pads, dil)
    ydt = _NAME_DT[y_dtype]
    if out is None:
        out = torch.empty((N, Ho, Wo, C), dtype=_DT_TORCH[ydt], device=x.device)
    _contig(out, "out")
    _check_out(out, (N, Ho, Wo), ydt)
    xq, wq, yq = _Q(x_scale, x_zp, 1), _per_tensor_or_channel(w_scale, w_zp), _Q(y_scale, y_zp, 1)
    _check(lib().qnn_depthwise_conv2d(_stream(stream), _ptr(x), _dt(x), N, H, W, C, xq.q, _ptr(w), R, S, wq.q,
                                      _ptr(bias), _cp(stride, pads, dil), _ptr(out), ydt, yq.q, _clamp(act),
                                      _ROUND[rounding], out.shape[-1], y_coff))
    return out


def dense(x: torch.Tensor, x_scale, x_zp, w: torch.Tensor, w_scale, w_zp, bias=None, y_scale=1.0, y_zp=0,
          y_dtype="i8", act=None, rounding="half_up", out: Optional[torch.Tensor] = None,
          stream=None) -> torch.Tensor:
    _contig(x, "x")
    _contig(w, "w")
    M, K = x.shape
    Nd = w.shape[0]
    ydt = _NAME_DT[y_dtype]
    if out is None:
        out = torch.empty((M, Nd), dtype=_DT_TORCH[ydt], device=x.device)
    _contig(out, "out")
    _check_out(out, (M,), ydt)
    xq, wq, yq = _Q(x_scale, x_zp, 1), _per_tensor_or_channel(w_scale, w_zp), _Q(y_scale, y_zp, 1)
    _check(lib().qnn_dense(_stream(stream), _ptr(x), _dt(x), M, K, xq.q, _ptr(w), Nd, wq.q, _ptr(bias),
                           _ptr(out), ydt, yq.q, _clamp(act), _ROUND[rounding], out.shape[-1]))
    return out


def requantize(x: torch.Tensor, x_scale, x_zp, y_scale, y_zp, y_dtype="u8", act=None, rounding="half_up",
               out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Standalone requantize; qparams per tensor or per innermost channel."""
    _contig(x, "x")
    channels = x.shape[-1] if x.dim() else 1
    ydt = _NAME_DT[y_dtype]
    if out is None:
        out = torch.empty(x.shape, dtype=_DT_TORCH[ydt], device=x.device)
    _contig(out, "out")
    _check_out(out, tuple(x.shape), ydt, whole=True)
    xq, yq = _per_tensor_or_channel(x_scale, x_zp), _per_tensor_or_channel(y_scale, y_zp)
    _check(lib().qnn_requantize(_stream(stream), _ptr(x), _dt(x), x.numel(), channels, xq.q, _ptr(out), ydt, yq.q,
                                _clamp(act), _ROUND[rounding]))
    return out


def add(a: torch.Tensor, a_scale, a_zp, b: torch.Tensor, b_scale, b_zp, y_scale, y_zp, y_dtype="u8", act=None,
        rounding="half_up", out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """qnn.add of two same-shape tensors with different per-tensor qparams."""
    _contig(a, "a")
    _contig(b, "b")
    if a.shape != b.shape:
        raise ValueError("add operands must have the same shape")
    ydt = _NAME_DT[y_dtype]
    if out is None:
        out = torch.empty(a.shape, dtype=_DT_TORCH[ydt], device=a.device)
    _contig(out, "out")
    _check_out(out, tuple(a.shape), ydt, whole=True)
    aq, bq, yq = _Q(a_scale, a_zp, 1), _Q(b_scale, b_zp, 1), _Q(y_scale, y_zp, 1)
    _check(lib().qnn_add(_stream(stream), _ptr(a), _dt(a), aq.q, _ptr(b), _dt(b), bq.q, a.numel(), _ptr(out), ydt,
                         yq.q, _clamp(act), _ROUND[rounding]))
    return out


_POOL_MODE = {"avg": 0, "max": 1}


def pool2d(x: torch.Tensor, mode="avg", kernel=(3, 3), stride=(1, 1), pads=0, count_pad=False, zp=0,
           rounding="half_away", out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Quantized pool2d of Eq. (4): NHWC u8/i8 in, same dtype out, scale and
    zero point unchanged.  "avg" rounds sum / count to nearest (ties by
    ``rounding``, "half_up" or "half_away"; padded cells count as ``zp`` when
    ``count_pad``), "max" takes the largest in-input cell.  Enqueued on the
    stream, no synchronization."""
    _contig(x, "x")
    if x.dim() != 4:
        raise ValueError("pool2d input must be NHWC")
    N, H, W, C = x.shape
    R, S = (kernel, kernel) if isinstance(kernel, int) else kernel
    cp = _cp(stride, pads, 1)
    Ho = (H + cp.pad_top + cp.pad_bottom - R) // cp.stride_h + 1
    Wo = (W + cp.pad_left + cp.pad_right - S) // cp.stride_w + 1
    if out is None:
        out = torch.empty((N, max(Ho, 0), max(Wo, 0), C), dtype=x.dtype, device=x.device)
    _contig(out, "out")
    if out.dtype != x.dtype or tuple(out.shape) != (N, Ho, Wo, C):
        raise ValueError(f"pool2d out must be {x.dtype} of shape {(N, Ho, Wo, C)}")
    _check(lib().qnn_pool2d(_stream(stream), _ptr(x), _dt(x), N, H, W, C, R, S, cp, _POOL_MODE[mode],
                            int(bool(count_pad)), int(zp), _ptr(out), _ROUND[rounding]))
    return out
