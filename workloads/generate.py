"""Seeded synthetic inputs shared by the oracle tests, the GPU parity tests and
the benchmark.  This module draws tensors and quantization parameters only;
it contains none of the quantized-operator arithmetic.

Recipe (values the workload descriptions leave open are fixed here):
  * numpy.random.default_rng(seed); draws in the order x, w, bias, qparams;
  * activations uint8 uniform over [0, 255]; weights int8, either uniform
    over [-127, 127] or rint(normal(0, sigma)) clipped to [-127, 127];
  * s_x = 0.02; per-channel s_w log-uniform over [1e-3, 1e-2];
  * output scale s_y = s_x * geomean(s_w) * sigma_acc / 48 rounded to binary32,
    with sigma_acc = sqrt(J * mean((x - zp_x)^2) * mean(w^2)) measured on the
    drawn tensors, so the median channel spans about +-48 output steps;
  * bias = rint(normal(0, sigma_acc / 4)) where a bias is used.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional, Tuple

import numpy as np

from .shapes import ConvLayer, DenseLayer, AddLayer, SINGLE_CONV

_NP = {"u8": np.uint8, "i8": np.int8, "i32": np.int32}
_RANGE = {"u8": (0, 255), "i8": (-128, 127)}


@dataclass
class ConvCase:
    """One quantized conv / depthwise / dense problem with all its parameters.

    Conv: x NHWC, w OHWI ([K][R][S][C]); depthwise: w [R][S][C]; dense: x [M][K]
    (stored as N=1, H=1, W=M), w [N][K] (stored as K, 1, 1, C).
    act is the (lo, hi) clamp in the output Q domain, or None."""
    name: str
    x: np.ndarray
    s_x: float
    zp_x: int
    w: np.ndarray
    s_w: np.ndarray
    zp_w: np.ndarray
    bias: Optional[np.ndarray]
    s_y: float
    zp_y: int
    yt: str = "u8"
    act: Optional[Tuple[int, int]] = None
    rounding: str = "half_up"
    stride: Tuple[int, int] = (1, 1)
    pads: Tuple[int, int, int, int] = (0, 0, 0, 0)
    depthwise: bool = False
    dense: bool = False
    # channel slice of a wider output tensor (concat): (offset, total channels)
    concat: Optional[Tuple[int, int]] = None

    @property
    def K(self):
        return self.w.shape[-1] if self.depthwise else self.w.shape[0]

    @property
    def J(self):
        if self.depthwise:
            return self.w.shape[0] * self.w.shape[1]
        return int(np.prod(self.w.shape[1:]))


@dataclass
class AddCase:
    name: str
    a: np.ndarray
    s_a: float
    zp_a: int
    b: np.ndarray
    s_b: float
    zp_b: int
    s_o: float
    zp_o: int
    yt: str = "u8"
    act: Optional[Tuple[int, int]] = None
    rounding: str = "half_up"


def _f32(v) -> float:
    return float(np.float32(v))


def _weights(rng, shape, sigma=None):
    if sigma is None:
        return rng.integers(-127, 128, size=shape, dtype=np.int8)
    w = np.rint(rng.normal(0.0, sigma, size=shape))
    return np.clip(w, -127, 127).astype(np.int8)


def _sigma_acc(x, zp_x, w, J):
    ex2 = float(np.mean((x.astype(np.float64) - zp_x) ** 2))
    ew2 = float(np.mean(w.astype(np.float64) ** 2))
    return float(np.sqrt(J * ex2 * max(ew2, 1e-12)))


def _output_scale(s_x, s_w, sigma_acc):
    gm = float(np.exp(np.mean(np.log(np.asarray(s_w, np.float64)))))
    return _f32(s_x * gm * max(sigma_acc, 1.0) / 48.0)


def _loguniform(rng, n, lo=1e-3, hi=1e-2):
    return (10.0 ** rng.uniform(np.log10(lo), np.log10(hi), size=n)).astype(np.float32)


def _act(kind, s_y, zp_y, yt):
    lo, hi = _RANGE[yt]
    if kind is None:
        return None
    if kind == "relu":
        return (max(lo, zp_y), hi)
    if kind == "relu6":
        return (max(lo, zp_y), min(hi, zp_y + int(np.rint(6.0 / s_y))))
    raise ValueError(kind)


def single_conv_case(seed: int = 1, s_y: float = 0.05) -> ConvCase:
    """14x14x64 3x3 stride-1 pad-1 conv at batch 1: x uniform uint8 with
    zp 128, s_x 0.02; w uniform int8 [-127, 127], per-tensor zp 0, s_w 0.005;
    uint8 output with s_y 0.05, zp 0; no bias; saturation only."""
    L = SINGLE_CONV
    rng = np.random.default_rng(seed)
    x = rng.integers(0, 256, size=(1, L.H, L.W, L.Cin), dtype=np.uint8)
    w = _weights(rng, (L.Cout, L.R, L.S, L.Cin))
    return ConvCase(L.name, x, 0.02, 128, w, np.array([0.005], np.float32),
                    np.zeros(1, np.int32), None, _f32(s_y), 0, "u8", None, "half_up",
                    (1, 1), L.pads)


def dense_case(layer: DenseLayer, seed: int, yt: str = "i8", zp_y: int = -3) -> ConvCase:
    """Dense: x uniform uint8 with zp 120, w rint(normal(0, 40)) clipped,
    per-output-channel log-uniform scales, zp_w 0, int8 output zp -3."""
    rng = np.random.default_rng(seed)
    x = rng.integers(0, 256, size=(layer.M, layer.K), dtype=np.uint8)
    w = _weights(rng, (layer.N, layer.K), sigma=40.0)
    s_x, zp_x = 0.02, 120
    s_w = _loguniform(rng, layer.N)
    s_y = _output_scale(s_x, s_w, _sigma_acc(x, zp_x, w, layer.K))
    return ConvCase(layer.name, x, s_x, zp_x, w, s_w, np.zeros(layer.N, np.int32), None,
                    s_y, zp_y, yt, None, "half_up", dense=True)


def conv_case(layer: ConvLayer, N: int, seed: int, *, act: Optional[str] = "auto",
              bias: bool = True, w_sigma: float = 30.0, zp_w: str = "zero",
              x_dtype: str = "u8", yt: str = "u8", rounding: str = "half_up",
              out_q: Optional[Tuple[float, int]] = None, w_dtype: str = "i8") -> ConvCase:
    """Conv / depthwise layer with asymmetric uint8 activations (random zp),
    per-channel int8 weights rint(normal(0, w_sigma)) clipped, random output
    zero point, and a ReLU clamp on layers followed by one.

    zp_w: "zero" (symmetric weights), "tensor" (one zp in [-20, 20]) or
    "channel" (per-channel zps in [-20, 20]).  out_q fixes (s_y, zp_y), e.g.
    the common output quantization of a concat group.  w_dtype "u8": asymmetric
    uint8 weights instead, zero points in [96, 160] (per tensor for zp_w
    "tensor", else per channel) and weights rint(normal(zp, w_sigma)) clipped
    to [0, 255]."""
    rng = np.random.default_rng(seed)
    if x_dtype == "u8":
        x = rng.integers(0, 256, size=(N, layer.H, layer.W, layer.Cin), dtype=np.uint8)
    else:
        x = rng.integers(-128, 128, size=(N, layer.H, layer.W, layer.Cin), dtype=np.int8)
    if layer.depthwise:
        w = _weights(rng, (layer.R, layer.S, layer.Cin), sigma=w_sigma)
        K, J = layer.Cin, layer.R * layer.S
    else:
        w = _weights(rng, (layer.Cout, layer.R, layer.S, layer.Cin), sigma=w_sigma)
        K, J = layer.Cout, layer.R * layer.S * layer.Cin
    lo, hi = _RANGE[x_dtype]
    zp_x = int(rng.integers(lo, hi + 1))
    s_x = 0.02
    s_w = _loguniform(rng, K)
    if w_dtype == "u8":
        zpw = (np.full(K, int(rng.integers(96, 161)), np.int32) if zp_w == "tensor"
               else rng.integers(96, 161, size=K).astype(np.int32))
        zc = zpw[None, None, :] if layer.depthwise else zpw[:, None, None, None]
        w = np.clip(np.rint(rng.normal(0.0, w_sigma, size=w.shape)) + zc, 0, 255).astype(np.uint8)
    elif zp_w == "zero":
        zpw = np.zeros(K, np.int32)
    elif zp_w == "tensor":
        zpw = np.full(K, int(rng.integers(-20, 21)), np.int32)
    elif zp_w == "channel":
        zpw = rng.integers(-20, 21, size=K).astype(np.int32)
    else:
        raise ValueError(zp_w)
    # spread of the weights about their zero point, for the output-scale rule
    wc = w.astype(np.int64) - (zpw[None, None, :] if layer.depthwise else zpw[:, None, None, None])
    sig = _sigma_acc(x, zp_x, wc, J)
    b = np.rint(rng.normal(0.0, sig / 4.0, size=K)).astype(np.int32) if bias else None
    if out_q is None:
        s_y = _output_scale(s_x, s_w, sig)
        zp_y = int(rng.integers(*_RANGE[yt])) if yt in _RANGE else 0
    else:
        s_y, zp_y = out_q
    if act == "auto":
        act = layer.act
    pads = layer.pads
    return ConvCase(layer.name, x, s_x, zp_x, w, s_w, zpw, b, s_y, zp_y, yt,
                    _act(act, s_y, zp_y, yt) if yt in _RANGE else None, rounding,
                    (layer.stride, layer.stride), pads, depthwise=layer.depthwise,
                    concat=None if layer.concat is None else layer.concat[1:])


def add_case(layer: AddLayer, N: int, seed: int, yt: str = "u8",
             rounding: str = "half_up") -> AddCase:
    """qnn.add of two uint8 NHWC tensors with independent (scale, zp)."""
    rng = np.random.default_rng(seed)
    shape = (N, layer.H, layer.W, layer.C)
    a = rng.integers(0, 256, size=shape, dtype=np.uint8)
    b = rng.integers(0, 256, size=shape, dtype=np.uint8)
    s_a, s_b = (_f32(v) for v in 10.0 ** rng.uniform(-2.5, -1.0, size=2))
    zp_a, zp_b = (int(v) for v in rng.integers(0, 256, size=2))
    s_o = _f32((s_a + s_b) * 1.1)
    zp_o = int(rng.integers(0, 256))
    return AddCase(layer.name, a, s_a, zp_a, b, s_b, zp_b, s_o, zp_o, yt, None, rounding)


def sample_indices(total: int, n: int, seed: int) -> np.ndarray:
    """Distinct sorted flat indices for sampled parity checks, always
    including the first and last elements."""
    rng = np.random.default_rng(seed)
    n = min(n, total)
    idx = rng.choice(total, size=n, replace=False) if total > n else np.arange(total)
    idx = np.union1d(idx, [0, total - 1])
    return idx.astype(np.int64)
