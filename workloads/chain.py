"""ResNet-50's conv body chained as in the network: the 7x7/2 stem, its 3x3/2
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

from .shapes import ConvLayer, resnet50


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
