"""Python front end of the CPU oracle (TEST INFRASTRUCTURE ONLY).

Only the tests, the smoke check and the CPU-baseline leg of the benchmark may
import this module.  It wraps ``libqnn_oracle.so`` (plain C int64 loop nests,
see ``qnn_oracle.c``) with numpy arrays and shares no code with the HIP
library.

Conventions (the same problem statement the paper gives, Sec. I-A Eq. (1),
Sec. II-B Eq. (2)/(3), Sec. III-B Eq. (5)):
  * activations NHWC, conv weights OHWI (row k holds R*S*C values, c fastest),
    depthwise weights [R][S][C], dense weights [N][K];
  * a quantized tensor is (Q, scale, zero_point); the weight scale and zero
    point are per tensor (length 1) or per output channel;
  * bias is int32 with implied scale s_x * s_w[k] and zero point 0;
  * rounding "half_up" (ties toward +inf), "half_away" (ties away from 0) or
    "two_stage" (for shifts of 31 or more: divide by 2^31 rounding half up,
    then by 2^(shift - 31) rounding half away from zero; Jacob et al.'s
    integer-only form).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libqnn_oracle.so")

DTYPE_CODE = {np.dtype(np.uint8): 0, np.dtype(np.int8): 1, np.dtype(np.int32): 2}
NAME_TO_NP = {"u8": np.uint8, "i8": np.int8, "i32": np.int32}
ROUNDING = {"half_up": 0, "half_away": 1, "two_stage": 2}
DTYPE_RANGE = {"u8": (0, 255), "i8": (-128, 127), "i32": (-(2**31), 2**31 - 1)}

_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _build

        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i32, i64, f32, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double
    lib.oracle_quantize_multiplier.argtypes = [f64, P, P]
    lib.oracle_quantize_multiplier.restype = ctypes.c_int
    lib.oracle_round_mul_shift.argtypes = [i64, i32, i32, ctypes.c_int]
    lib.oracle_round_mul_shift.restype = i64
    lib.oracle_requantize_value.argtypes = [i64, f64, i32, i32, i64, i64, i32, P]
    lib.oracle_requantize_value.restype = ctypes.c_int
    lib.oracle_pool2d.argtypes = [P, i32, P, P, i32, i32, i32, i32, P]
    lib.oracle_pool2d.restype = ctypes.c_int
    lib.oracle_conv_out_hw.argtypes = [P, P, P, P]
    lib.oracle_conv_out_hw.restype = None
    lib.oracle_conv2d_acc.argtypes = [P, i32, i32, P, i32, P, P, P, P, i32, P]
    lib.oracle_conv2d_acc.restype = None
    lib.oracle_conv2d_acc_points.argtypes = [P, i32, i32, P, i32, P, P, P, P, i32, P, i64, P]
    lib.oracle_conv2d_acc_points.restype = None
    lib.oracle_dense_acc.argtypes = [P, i32, i32, P, i32, P, P, i64, i64, i64, P]
    lib.oracle_dense_acc.restype = None
    lib.oracle_requantize_acc.argtypes = [P, i64, i64, f32, P, i32, f32, i32, i32,
                                          i64, i64, i32, P, i64, i64]
    lib.oracle_requantize_acc.restype = ctypes.c_int
    lib.oracle_requantize_points.argtypes = [P, P, i64, i64, f32, P, i32, f32, i32,
                                             i32, i64, i64, i32, P]
    lib.oracle_requantize_points.restype = ctypes.c_int
    lib.oracle_requantize.argtypes = [P, i32, i64, i64, P, P, i32, P, P, i32, i32,
                                      i64, i64, i32, P]
    lib.oracle_requantize.restype = ctypes.c_int
    lib.oracle_add.argtypes = [P, i32, f32, i32, P, i32, f32, i32, i64, f32, i32, i32,
                               i64, i64, i32, P]
    lib.oracle_add.restype = ctypes.c_int
    lib.oracle_threads.restype = ctypes.c_int
    lib.oracle_set_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_threads.restype = None
    _lib = lib
    return lib


def threads() -> int:
    """OpenMP threads the oracle's loops run on."""
    return int(_load().oracle_threads())


def set_threads(n: int) -> None:
    """Run the oracle's later loops on n threads (timing only)."""
    _load().oracle_set_threads(int(n))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _per_channel(v, n, dtype):
    a = np.atleast_1d(np.asarray(v, dtype=dtype))
    if a.size not in (1, n):
        raise ValueError(f"per-channel parameter has {a.size} entries, expected 1 or {n}")
    return np.ascontiguousarray(np.broadcast_to(a, (n,)) if a.size == 1 else a, dtype=dtype)


def _clamp_bounds(yt, act):
    lo, hi = DTYPE_RANGE[yt]
    if act is not None:
        lo, hi = max(lo, act[0]), min(hi, act[1])
    return lo, hi


# --------------------------------------------------------------------------
# scalar requantize pieces (Eq. (5) with a fixed-point multiplier)
# --------------------------------------------------------------------------

def quantize_multiplier(M: float):
    """(mult, shift) with M ~= mult * 2**-shift, mult in [2^30, 2^31)."""
    lib = _load()
    m, s = ctypes.c_int32(), ctypes.c_int32()
    if lib.oracle_quantize_multiplier(float(M), ctypes.byref(m), ctypes.byref(s)) != 0:
        raise ValueError(f"multiplier {M!r} is outside the representable range")
    return m.value, s.value


def round_mul_shift(v: int, mult: int, shift: int, rounding: str = "half_up") -> int:
    return int(_load().oracle_round_mul_shift(int(v), int(mult), int(shift), ROUNDING[rounding]))


def requantize_value(v: int, M: float, zp_out: int = 0, yt: str = "i32",
                     act=None, rounding: str = "half_up") -> int:
    lo, hi = _clamp_bounds(yt, act)
    out = ctypes.c_int64()
    rc = _load().oracle_requantize_value(int(v), float(M), int(zp_out), DTYPE_CODE[np.dtype(NAME_TO_NP[yt])],
                                         lo, hi, ROUNDING[rounding], ctypes.byref(out))
    if rc != 0:
        raise ValueError("requantize outside its domain")
    return out.value


# --------------------------------------------------------------------------
# accumulators (Eq. (2)/(3) product form, zero-point padding, bias)
# --------------------------------------------------------------------------

def conv_out_hw(H, W, R, S, stride=(1, 1), pads=(0, 0, 0, 0), dil=(1, 1)):
    shape = _c([1, H, W, 1, 1, R, S], np.int32)
    cp = _c([stride[0], stride[1], pads[0], pads[1], pads[2], pads[3], dil[0], dil[1]], np.int32)
    ho, wo = ctypes.c_int64(), ctypes.c_int64()
    _load().oracle_conv_out_hw(_ptr(shape), _ptr(cp), ctypes.byref(ho), ctypes.byref(wo))
    return ho.value, wo.value


def _weights(w):
    """Weights as given when uint8 (asymmetric uint8 weights), else int8."""
    w = np.ascontiguousarray(w)
    return w if w.dtype == np.uint8 else _c(w, np.int8)


def _conv_args(x, w, zp_w, bias, stride, pads, dil, depthwise):
    x = np.ascontiguousarray(x)
    if x.dtype not in DTYPE_CODE or x.dtype == np.int32:
        raise TypeError("activations must be uint8 or int8")
    w = _weights(w)
    N, H, W, C = x.shape
    if depthwise:
        R, S, Cw = w.shape
        if Cw != C:
            raise ValueError("depthwise weight channels != input channels")
        K = C
    else:
        K, R, S, Cw = w.shape
        if Cw != C:
            raise ValueError("weight Cin != input C")
    zpw = _per_channel(zp_w, K, np.int32)
    b = None if bias is None else _c(bias, np.int32)
    if b is not None and b.shape != (K,):
        raise ValueError("bias must have one entry per output channel")
    # pads = (top, left, bottom, right)
    shape = _c([N, H, W, C, K, R, S], np.int32)
    cp = _c([stride[0], stride[1], pads[0], pads[1], pads[2], pads[3], dil[0], dil[1]], np.int32)
    return x, w, zpw, b, shape, cp, (N, H, W, C, K, R, S)


def conv2d_acc(x, zp_x, w, zp_w=0, bias=None, stride=(1, 1), pads=(0, 0, 0, 0),
               dil=(1, 1), depthwise=False):
    """int64 accumulators acc[n, oh, ow, k] including bias (no requantize)."""
    x, w, zpw, b, shape, cp, dims = _conv_args(x, w, zp_w, bias, stride, pads, dil, depthwise)
    N, H, W, C, K, R, S = dims
    Ho, Wo = conv_out_hw(H, W, R, S, stride, pads, dil)
    acc = np.empty((N, Ho, Wo, K), np.int64)
    _load().oracle_conv2d_acc(_ptr(x), DTYPE_CODE[x.dtype], int(zp_x), _ptr(w), DTYPE_CODE[w.dtype], _ptr(zpw),
                              _ptr(b), _ptr(shape), _ptr(cp), int(bool(depthwise)), _ptr(acc))
    return acc


def conv2d_acc_points(x, zp_x, w, idx, zp_w=0, bias=None, stride=(1, 1),
                      pads=(0, 0, 0, 0), dil=(1, 1), depthwise=False):
    """Accumulators at flat output indices idx = ((n*Ho + oh)*Wo + ow)*K + k."""
    x, w, zpw, b, shape, cp, _ = _conv_args(x, w, zp_w, bias, stride, pads, dil, depthwise)
    idx = _c(idx, np.int64)
    acc = np.empty(idx.shape, np.int64)
    _load().oracle_conv2d_acc_points(_ptr(x), DTYPE_CODE[x.dtype], int(zp_x), _ptr(w), DTYPE_CODE[w.dtype],
                                     _ptr(zpw),
                                     _ptr(b), _ptr(shape), _ptr(cp), int(bool(depthwise)),
                                     _ptr(idx), idx.size, _ptr(acc))
    return acc


def dense_acc(x, zp_x, w, zp_w=0, bias=None):
    """int64 acc[m, n] = bias[n] + sum_k (x[m,k]-zp_x) * (w[n,k]-zp_w[n])."""
    x = np.ascontiguousarray(x)
    w = _weights(w)
    M, Kd = x.shape
    Nd, Kw = w.shape
    if Kw != Kd:
        raise ValueError("dense K mismatch")
    zpw = _per_channel(zp_w, Nd, np.int32)
    b = None if bias is None else _c(bias, np.int32)
    acc = np.empty((M, Nd), np.int64)
    _load().oracle_dense_acc(_ptr(x), DTYPE_CODE[x.dtype], int(zp_x), _ptr(w), DTYPE_CODE[w.dtype], _ptr(zpw),
                             _ptr(b),
                             M, Kd, Nd, _ptr(acc))
    return acc


# --------------------------------------------------------------------------
# requantize of accumulators, and the fused ops built from the pieces
# --------------------------------------------------------------------------

def requantize_acc(acc, s_x, s_w, s_y, zp_y, yt="u8", act=None, rounding="half_up",
                   out=None, y_ldc=None, y_coff=0):
    """Requantize acc[..., K] with M_k = s_x*s_w[k]/s_y (Eq. (5)).

    With ``out`` given, element (m, k) is written to out.flat[m*y_ldc + y_coff + k]
    (a channel slice of a wider NHWC tensor, as in a concat)."""
    acc = _c(acc, np.int64)
    K = acc.shape[-1]
    rows = acc.size // K
    sw = np.atleast_1d(_c(s_w, np.float32))
    if sw.size not in (1, K):
        raise ValueError("s_w must be per tensor or per output channel")
    if out is None:
        out = np.zeros(acc.shape, NAME_TO_NP[yt])
        y_ldc = K
    if y_ldc is None:
        raise ValueError("y_ldc required with out")
    lo, hi = _clamp_bounds(yt, act)
    rc = _load().oracle_requantize_acc(_ptr(acc), rows, K, float(s_x), _ptr(sw), sw.size,
                                       float(s_y), int(zp_y), DTYPE_CODE[np.dtype(NAME_TO_NP[yt])],
                                       lo, hi, ROUNDING[rounding], _ptr(out), int(y_ldc), int(y_coff))
    if rc != 0:
        raise ValueError("invalid requantize multiplier")
    return out


def requantize_points(acc, idx, K, s_x, s_w, s_y, zp_y, yt="u8", act=None, rounding="half_up"):
    acc = _c(acc, np.int64)
    idx = _c(idx, np.int64)
    sw = np.atleast_1d(_c(s_w, np.float32))
    lo, hi = _clamp_bounds(yt, act)
    out = np.empty(acc.shape, np.int64)
    rc = _load().oracle_requantize_points(_ptr(acc), _ptr(idx), idx.size, int(K), float(s_x), _ptr(sw),
                                          sw.size, float(s_y), int(zp_y),
                                          DTYPE_CODE[np.dtype(NAME_TO_NP[yt])], lo, hi,
                                          ROUNDING[rounding], _ptr(out))
    if rc != 0:
        raise ValueError("invalid requantize multiplier")
    return out


def conv2d(x, s_x, zp_x, w, s_w, zp_w, bias, s_y, zp_y, yt="u8", act=None,
           rounding="half_up", stride=(1, 1), pads=(0, 0, 0, 0), dil=(1, 1),
           depthwise=False):
    """qnn.conv2d -> bias_add -> requantize -> clamp, NHWC output."""
    acc = conv2d_acc(x, zp_x, w, zp_w, bias, stride, pads, dil, depthwise)
    if yt == "i32":
        return acc.astype(np.int32)
    return requantize_acc(acc, s_x, s_w, s_y, zp_y, yt, act, rounding)


def dense(x, s_x, zp_x, w, s_w, zp_w, bias, s_y, zp_y, yt="i8", act=None, rounding="half_up"):
    acc = dense_acc(x, zp_x, w, zp_w, bias)
    if yt == "i32":
        return acc.astype(np.int32)
    return requantize_acc(acc, s_x, s_w, s_y, zp_y, yt, act, rounding)


def requantize(x, s_in, zp_in, s_out, zp_out, yt="u8", act=None, rounding="half_up"):
    """Standalone requantize; qparams per tensor or per innermost channel."""
    x = np.ascontiguousarray(x)
    C = x.shape[-1] if x.ndim else 1
    si = np.atleast_1d(_c(s_in, np.float32))
    zi = np.atleast_1d(_c(zp_in, np.int32))
    so = np.atleast_1d(_c(s_out, np.float32))
    zo = np.atleast_1d(_c(zp_out, np.int32))
    if si.size != zi.size or so.size != zo.size:
        raise ValueError("scale and zero point must have the same length")
    y = np.empty(x.shape, NAME_TO_NP[yt])
    lo, hi = _clamp_bounds(yt, act)
    rc = _load().oracle_requantize(_ptr(x), DTYPE_CODE[x.dtype], x.size, C, _ptr(si), _ptr(zi), si.size,
                                   _ptr(so), _ptr(zo), so.size, DTYPE_CODE[np.dtype(NAME_TO_NP[yt])],
                                   lo, hi, ROUNDING[rounding], _ptr(y))
    if rc != 0:
        raise ValueError("requantize outside its domain")
    return y


def add(a, s_a, zp_a, b, s_b, zp_b, s_o, zp_o, yt="u8", act=None, rounding="half_up"):
    """qnn.add of two differently scaled tensors of the same shape."""
    a = np.ascontiguousarray(a)
    b = np.ascontiguousarray(b)
    if a.shape != b.shape:
        raise ValueError("add operands must have the same shape")
    y = np.empty(a.shape, NAME_TO_NP[yt])
    lo, hi = _clamp_bounds(yt, act)
    rc = _load().oracle_add(_ptr(a), DTYPE_CODE[a.dtype], float(s_a), int(zp_a), _ptr(b),
                            DTYPE_CODE[b.dtype], float(s_b), int(zp_b), a.size, float(s_o), int(zp_o),
                            DTYPE_CODE[np.dtype(NAME_TO_NP[yt])], lo, hi, ROUNDING[rounding], _ptr(y))
    if rc != 0:
        raise ValueError("invalid add multipliers")
    return y


POOL_MODES = {"avg": 0, "max": 1}


def pool2d(x, mode="avg", kernel=(3, 3), stride=(1, 1), pads=(0, 0, 0, 0), count_pad=False, zp=0,
           rounding="half_away"):
    """Quantized pool2d, Eq. (4): scale and zero point pass through, the
    quantized input is pooled.  x NHWC u8/i8; pads (top, left, bottom, right);
    "avg" rounds sum / count to nearest (ties by ``rounding``: "half_up" or
    "half_away"), counting padded cells as ``zp`` when ``count_pad``; "max"
    takes the largest in-input cell.  Returns the NHWC output, x's dtype."""
    if rounding not in ("half_up", "half_away"):
        raise ValueError("pool2d rounding is half_up or half_away")
    x = np.ascontiguousarray(x)
    N, H, W, C = x.shape
    R, S = kernel
    sh, sw = stride
    pt, pl, pb, pr = pads
    Ho, Wo = (H + pt + pb - R) // sh + 1, (W + pl + pr - S) // sw + 1
    y = np.zeros((N, max(Ho, 0), max(Wo, 0), C), dtype=x.dtype)
    shape = np.array([N, H, W, C, R, S], np.int32)
    pp = np.array([sh, sw, pt, pl, pb, pr], np.int32)
    rc = _load().oracle_pool2d(_ptr(x), DTYPE_CODE[x.dtype], _ptr(shape), _ptr(pp), POOL_MODES[mode],
                               int(bool(count_pad)), int(zp), ROUNDING[rounding], _ptr(y))
    if rc != 0:
        raise ValueError("pool2d: a window holds no input cell")
    return y
