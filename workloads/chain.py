"""Networks chained as they run, with int8 hand-off between steps.

ResNet-50's conv body: the 7x7/2 stem, its 3x3/2
max pool, the 16 bottleneck blocks and the global 7x7 average pool.  Every
step reads the int8 tensor its producer wrote, with the producer's (scale,
zero point), every block ends in a qnn.add of its main path and its shortcut
(the block input, or the projection conv of the first block of a stage), and
pooling keeps its input's (scale, zero point) (Eq. (4)).
Only shapes and quantization parameters are drawn here; this module holds no
quantized-operator arithmetic.

Recipe (numpy.random.default_rng(seed), drawn in the order below):
  * input x0: an int8 image N x 224 x 224 x 3, uniform over [-128, 127],
    scale 0.02, zero point -10;
  * per conv, in layer order: weights rint(normal(0, 30)) clipped to
    [-127, 127], per-channel scales log-uniform over one decade centred on
    48 / sigma_acc (so that an output scale stays near its input's through
    the 68 steps), weight zero points 0, bias rint(normal(0, sigma_acc / 4));
    sigma_acc = sqrt(J * E[(x - zp_x)^2] * mean(w^2)), E[(x - zp_x)^2] taken
    as 48^2 for a linear producer and 48^2 / 2 after a ReLU (half the
    values sit on the zero point), and measured on x0;
  * output scale by the rule of ``generate.py`` (median channel about +-48
    output steps): s_y = s_x * geomean(s_w) * sigma_acc / 48;
  * zero points: -100 for outputs followed by a ReLU (the clamp keeps
    [-100, 127]), 0 for the linear 1x1b and projection outputs;
  * add: output scale 1.5 x the larger input scale, zero point -100, ReLU;
  * pools: max 3x3/2 with pads 1 after the stem, average 7x7 (rounding half
    away from zero) after the last block.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Tuple, Union

import numpy as np

from .shapes import ConvLayer, inception_v3, mobilenet_v2_blocks, resnet50


@dataclass
class ChainConv:
    layer: ConvLayer
    src: str
    dst: str
    w: np.ndarray            # int8 OHWI
    s_w: np.ndarray
    zp_w: np.ndarray
    bias: np.ndarray         # int32 [K]
    s_y: float
    zp_y: int
    act: Optional[Tuple[int, int]]
    # channel slice of a concat tensor the conv writes: (offset, total channels)
    y_off: Optional[Tuple[int, int]] = None


@dataclass
class ChainAdd:
    name: str
    a: str
    b: str
    dst: str
    s_o: float
    zp_o: int
    act: Optional[Tuple[int, int]]


@dataclass
class ChainPool:
    name: str
    src: str
    dst: str
    mode: str                            # "max" or "avg"
    kernel: Tuple[int, int]
    stride: Tuple[int, int]
    pads: Tuple[int, int, int, int]


@dataclass
class Chain:
    x0: np.ndarray                       # int8 NHWC image
    q: dict                              # tensor name -> (scale, zero point)
    steps: List[Union[ChainConv, ChainAdd, ChainPool]]
    N: int

    def graph(self):
        """The steps as (kind, input names, output name): "conv" for a conv
        writing a whole tensor, "conv_slice" for one writing a concat's
        channel slice, "dw", "pool" and "add"."""
        out = []
        for st in self.steps:
            if isinstance(st, ChainConv):
                kind = "dw" if st.layer.depthwise else ("conv" if st.y_off is None else "conv_slice")
                out.append((kind, (st.src,), st.dst))
            elif isinstance(st, ChainPool):
                out.append(("pool", (st.src,), st.dst))
            else:
                out.append(("add", (st.a, st.b), st.dst))
        return out


def _f32(v) -> float:
    return float(np.float32(v))


def resnet50_chain(N: int, seed: int = 6000) -> Chain:
    rng = np.random.default_rng(seed)
    stem = [l for l in resnet50() if l.name.startswith("stem")][0]
    layers = [l for l in resnet50() if not l.name.startswith("stem")]
    x0 = rng.integers(-128, 128, size=(N, 224, 224, 3), dtype=np.int8)
    q = {"x0": (0.02, -10)}
    spread2 = {"x0": float(np.mean((x0.astype(np.float64) + 10.0) ** 2))}
    steps: List[Union[ChainConv, ChainAdd, ChainPool]] = []

    def conv(layer: ConvLayer, src: str, dst: str):
        s_x, _ = q[src]
        w = np.clip(np.rint(rng.normal(0.0, 30.0, size=(layer.Cout, layer.R, layer.S, layer.Cin))),
                    -127, 127).astype(np.int8)
        J = layer.R * layer.S * layer.Cin
        sig = float(np.sqrt(J * spread2[src] * float(np.mean(w.astype(np.float64) ** 2))))
        s_w = (48.0 / sig * 10.0 ** rng.uniform(-0.5, 0.5, size=layer.Cout)).astype(np.float32)
        bias = np.rint(rng.normal(0.0, sig / 4.0, size=layer.Cout)).astype(np.int32)
        gm = float(np.exp(np.mean(np.log(s_w.astype(np.float64)))))
        s_y = _f32(s_x * gm * max(sig, 1.0) / 48.0)
        relu = layer.act == "relu"
        zp_y = -100 if relu else 0
        q[dst] = (s_y, zp_y)
        spread2[dst] = 48.0 ** 2 / 2 if relu else 48.0 ** 2
        steps.append(ChainConv(layer, src, dst, w, s_w, np.zeros(layer.Cout, np.int32), bias, s_y, zp_y,
                               (zp_y, 127) if relu else None))

    def pool(name, src, dst, mode, kernel, stride, pads):
        q[dst] = q[src]
        spread2[dst] = spread2[src]
        steps.append(ChainPool(name, src, dst, mode, kernel, stride, pads))

    conv(stem, "x0", "stem")
    pool("stem_pool", "stem", "pool", "max", (3, 3), (2, 2), (1, 1, 1, 1))
    cur = "pool"
    i = 0
    while i < len(layers):
        pre = layers[i].name.split("_")[0]
        block = [l for l in layers[i:i + 4] if l.name.startswith(pre + "_")]
        byname = {l.name.split("_")[1]: l for l in block}
        conv(byname["1x1a"], cur, pre + "_a")
        conv(byname["3x3"], pre + "_a", pre + "_b")
        conv(byname["1x1b"], pre + "_b", pre + "_c")
        short = cur
        if "proj" in byname:
            conv(byname["proj"], cur, pre + "_p")
            short = pre + "_p"
        s_o = _f32(1.5 * max(q[pre + "_c"][0], q[short][0]))
        q[pre + "_out"] = (s_o, -100)
        spread2[pre + "_out"] = 48.0 ** 2 / 2
        steps.append(ChainAdd(pre + "_add", pre + "_c", short, pre + "_out", s_o, -100, (-100, 127)))
        cur = pre + "_out"
        i += len(block)
    pool("gap", cur, "gap", "avg", (7, 7), (1, 1), (0, 0, 0, 0))
    return Chain(x0, q, steps, N)


class _Builder:
    """Draws the weights and quantization of chained convs (recipe of the
    module docstring), tracking each tensor's (scale, zero point) and the
    mean square of its values about the zero point."""

    def __init__(self, rng, x0, s0, zp0):
        self.rng = rng
        self.q = {"x0": (s0, zp0)}
        self.spread2 = {"x0": float(np.mean((x0.astype(np.float64) - zp0) ** 2))}
        self.steps: List[Union[ChainConv, ChainAdd, ChainPool]] = []

    def draw(self, layer: ConvLayer, src: str):
        """Weights, scales and bias of a conv reading src, and the output
        scale the rule gives it."""
        rng = self.rng
        shape = (layer.R, layer.S, layer.Cin) if layer.depthwise else (layer.Cout, layer.R, layer.S, layer.Cin)
        w = np.clip(np.rint(rng.normal(0.0, 30.0, size=shape)), -127, 127).astype(np.int8)
        J = layer.R * layer.S * (1 if layer.depthwise else layer.Cin)
        sig = float(np.sqrt(J * self.spread2[src] * float(np.mean(w.astype(np.float64) ** 2))))
        s_w = (48.0 / sig * 10.0 ** rng.uniform(-0.5, 0.5, size=layer.Cout)).astype(np.float32)
        bias = np.rint(rng.normal(0.0, sig / 4.0, size=layer.Cout)).astype(np.int32)
        gm = float(np.exp(np.mean(np.log(s_w.astype(np.float64)))))
        s_y = _f32(self.q[src][0] * gm * max(sig, 1.0) / 48.0)
        return w, s_w, bias, s_y

    def conv(self, layer: ConvLayer, src: str, dst: str, drawn=None, out_q=None, y_off=None):
        w, s_w, bias, s_y = drawn if drawn is not None else self.draw(layer, src)
        act_kind = layer.act
        zp_y = -100 if act_kind in ("relu", "relu6") else 0
        if out_q is not None:
            s_y, zp_y = out_q
        act = None
        if act_kind == "relu":
            act = (zp_y, 127)
        elif act_kind == "relu6":
            act = (zp_y, int(min(127, zp_y + np.rint(6.0 / s_y))))
        self.q[dst] = (s_y, zp_y)
        self.spread2[dst] = 48.0 ** 2 / 2 if act_kind else 48.0 ** 2
        self.steps.append(ChainConv(layer, src, dst, w, s_w, np.zeros(layer.Cout, np.int32), bias, s_y, zp_y,
                                    act, y_off))

    def add(self, name, a, b, dst, relu):
        s_o = _f32(1.5 * max(self.q[a][0], self.q[b][0]))
        zp = -100 if relu else 0
        self.q[dst] = (s_o, zp)
        self.spread2[dst] = 48.0 ** 2 / 2 if relu else 48.0 ** 2
        self.steps.append(ChainAdd(name, a, b, dst, s_o, zp, (-100, 127) if relu else None))

    def pool(self, name, src, dst, mode, kernel, stride, pads):
        self.q[dst] = self.q[src]
        self.spread2[dst] = self.spread2[src]
        self.steps.append(ChainPool(name, src, dst, mode, kernel, stride, pads))


def mobilenet_v2_chain(N: int, seed: int = 6100) -> Chain:
    """MobileNet-V2's expansion-6 inverted residuals chained as in the
    network, from the 112 x 112 x 16 tensor the expansion-1 first block
    produces (an int8 input here, uniform, scale 0.02, zero point 0): per
    block a 1x1 expand (ReLU6), a 3x3 depthwise (stride 1 or 2, ReLU6) and a
    linear 1x1 project, plus a qnn.add of the block input (output scale 1.5 x
    the larger input scale, zero point 0, no clamp) when the stride is 1 and
    the widths match; ReLU6 outputs have zero point -100 and the upper clamp
    at -100 + rint(6 / scale) (at most 127); weights and scales as in
    resnet50_chain.  17 blocks, 51 convs, 10 adds."""
    rng = np.random.default_rng(seed)
    x0 = rng.integers(-128, 128, size=(N, 112, 112, 16), dtype=np.int8)
    B = _Builder(rng, x0, 0.02, 0)
    cur = "x0"
    for blk in mobilenet_v2_blocks():
        ho = blk.H // blk.stride
        pads = (1, 1, 1, 1) if blk.stride == 1 else (0, 0, 1, 1)
        B.conv(ConvLayer(f"{blk.name}_expand", blk.H, blk.H, blk.Cin, blk.hidden, 1, 1, act="relu6"), cur,
               blk.name + "_e")
        B.conv(ConvLayer(f"{blk.name}_dw", blk.H, blk.H, blk.hidden, blk.hidden, 3, 3, blk.stride, pads,
                         depthwise=True, act="relu6"), blk.name + "_e", blk.name + "_d")
        B.conv(ConvLayer(f"{blk.name}_project", ho, ho, blk.hidden, blk.Cout, 1, 1, act=None), blk.name + "_d",
               blk.name + "_p")
        if blk.residual:
            B.add(blk.name + "_add", blk.name + "_p", cur, blk.name + "_out", relu=False)
            cur = blk.name + "_out"
        else:
            cur = blk.name + "_p"
    return Chain(x0, B.q, B.steps, N)


def inception_v3_mixed5_chain(N: int, seed: int = 6200) -> Chain:
    """Inception-v3's Mixed 5b and 5c chained as in the network, from the
    35 x 35 x 192 tensor the stem produces (an int8 input here, uniform,
    scale 0.02, zero point 0).  Per block four branches read the block
    input: 1x1; 1x1 then 5x5; 1x1 then two 3x3; a 3x3/1 average pool (pads
    1, padded cells left out, Eq. (4)) then 1x1.  The last conv of each
    branch writes its channel slice of the block output with the block's
    common (scale, zero point): the largest output scale the rule gives the
    four, zero point -100, ReLU.  Weights and inner scales as in
    resnet50_chain.  14 convs, 2 pools, 2 concats."""
    rng = np.random.default_rng(seed)
    x0 = rng.integers(-128, 128, size=(N, 35, 35, 192), dtype=np.int8)
    B = _Builder(rng, x0, 0.02, 0)
    cur = "x0"
    layers = {l.name: l for l in inception_v3()}
    for tag in ("5b", "5c"):
        g = f"mixed{tag}"
        L = lambda n: layers[f"{g}_{n}"]   # noqa: E731
        total = L("b1_1x1").concat[2]
        B.pool(f"{g}_pool", cur, f"{g}_pooled", "avg", (3, 3), (1, 1), (1, 1, 1, 1))
        B.conv(L("b2_1x1"), cur, f"{g}_b2a")
        B.conv(L("b3_1x1"), cur, f"{g}_b3a")
        B.conv(L("b3_3x3a"), f"{g}_b3a", f"{g}_b3b")
        finals = [("b1_1x1", cur), ("b2_5x5", f"{g}_b2a"), ("b3_3x3b", f"{g}_b3b"), ("b4_1x1", f"{g}_pooled")]
        drawn = [B.draw(L(n), src) for n, src in finals]
        common = (max(d[3] for d in drawn), -100)
        for (n, src), d in zip(finals, drawn):
            B.conv(L(n), src, g, drawn=d, out_q=common, y_off=(L(n).concat[1], total))
        cur = g
    return Chain(x0, B.q, B.steps, N)
