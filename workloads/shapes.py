"""Layer shape tables of the synthetic workloads (shapes only, no arithmetic).

The paper evaluates pre-quantized ImageNet CNNs at batch 1 (Sec. IV-A/IV-C):
ResNet, MobileNet and Inception families.  Their trained weights and the
dataset are not available here; these tables reproduce only the layer
shapes of the published architectures, so that seeded synthetic tensors of
the same shapes can stand in for them.

Every conv entry lists its input spatial size explicitly, so no output-size
arithmetic happens here.  Fields: name, H, W, Cin, Cout, R, S, stride,
pads (top, left, bottom, right).
"""
from dataclasses import dataclass, field
from typing import List, Optional, Tuple


@dataclass(frozen=True)
class ConvLayer:
    name: str
    H: int
    W: int
    Cin: int
    Cout: int
    R: int
    S: int
    stride: int = 1
    pads: Tuple[int, int, int, int] = (0, 0, 0, 0)
    depthwise: bool = False
    act: Optional[str] = "relu"  # clamp after requantize: "relu", "relu6" or None
    # channel slice of a concat output this layer writes (Inception blocks)
    concat: Optional[Tuple[str, int, int]] = None  # (group, channel offset, total channels)


@dataclass(frozen=True)
class DenseLayer:
    name: str
    M: int
    K: int
    N: int


@dataclass(frozen=True)
class AddLayer:
    name: str
    H: int
    W: int
    C: int


def _same(k):
    p = k // 2
    return (p, p, p, p)


# ---------------------------------------------------------------- ResNet-50 v1.5
def resnet50() -> List[ConvLayer]:
    """Stem 7x7/2 and the 16 bottlenecks (3, 4, 6, 3) with the stride on the
    first 3x3 of stages 2-4, plus the 4 projection shortcuts (53 convs)."""
    L = [ConvLayer("stem7x7s2", 224, 224, 3, 64, 7, 7, 2, (3, 3, 3, 3))]
    stages = [(56, 64, 256, 3), (28, 128, 512, 4), (14, 256, 1024, 6), (7, 512, 2048, 3)]
    cin = 64
    in_hw = 56
    for si, (hw, width, cout, blocks) in enumerate(stages):
        for b in range(blocks):
            pre = f"s{hw}b{b}"
            first = b == 0
            stride = 2 if (first and si > 0) else 1
            h_in = in_hw if first else hw
            L.append(ConvLayer(f"{pre}_1x1a", h_in, h_in, cin, width, 1, 1))
            L.append(ConvLayer(f"{pre}_3x3", h_in, h_in, width, width, 3, 3, stride, (1, 1, 1, 1)))
            L.append(ConvLayer(f"{pre}_1x1b", hw, hw, width, cout, 1, 1, act=None))
            if first:
                L.append(ConvLayer(f"{pre}_proj", h_in, h_in, cin, cout, 1, 1, stride, act=None))
            cin = cout
        in_hw = hw
    return L


# ---------------------------------------------------------------- MobileNet-V2
@dataclass(frozen=True)
class InvertedResidual:
    name: str
    H: int
    Cin: int
    Cout: int
    stride: int
    expand: int = 6

    @property
    def hidden(self):
        return self.Cin * self.expand

    @property
    def residual(self):
        return self.stride == 1 and self.Cin == self.Cout


def mobilenet_v2_blocks() -> List[InvertedResidual]:
    """The expansion-6 inverted residual blocks, (c, n, s) = (24,2,2), (32,3,2),
    (64,4,2), (96,3,1), (160,3,2), (320,1,1); input 112x112x16 after the stem
    and the expansion-1 first block."""
    spec = [(24, 2, 2), (32, 3, 2), (64, 4, 2), (96, 3, 1), (160, 3, 2), (320, 1, 1)]
    blocks = []
    cin, hw = 16, 112
    for c, n, s in spec:
        for i in range(n):
            stride = s if i == 0 else 1
            blocks.append(InvertedResidual(f"c{c}_{i}", hw, cin, c, stride))
            if stride == 2:
                hw = (hw + 1) // 2
            cin = c
    return blocks


def mobilenet_v2_layers():
    """Flattened per-block layers: 1x1 expand (ReLU6), 3x3 depthwise (ReLU6),
    1x1 project (linear), optional residual add.  Input sizes are listed per
    block from the architecture (112 -> 56 -> 28 -> 14 -> 7)."""
    out = []
    for b in mobilenet_v2_blocks():
        h_out = b.H // b.stride
        out.append(ConvLayer(f"{b.name}_expand", b.H, b.H, b.Cin, b.hidden, 1, 1, act="relu6"))
        out.append(ConvLayer(f"{b.name}_dw", b.H, b.H, b.hidden, b.hidden, 3, 3, b.stride,
                             (1, 1, 1, 1) if b.stride == 1 else (0, 0, 1, 1), depthwise=True,
                             act="relu6"))
        out.append(ConvLayer(f"{b.name}_project", h_out, h_out, b.hidden, b.Cout, 1, 1, act=None))
        if b.residual:
            out.append(AddLayer(f"{b.name}_add", h_out, h_out, b.Cout))
    return out


# ---------------------------------------------------------------- Inception-v3
def inception_v3() -> List[ConvLayer]:
    """The 94 convolutions of Inception-v3 at 299x299 (stem, Mixed 5b-5d, 6a,
    6b-6e, 7a, 7b-7c).  Branch convs that end a block carry the concat slice
    they write; pooling layers are not part of the conv path and are omitted
    (the 1x1 convs of the pooling branches run on pooled-shape inputs)."""
    L = [
        ConvLayer("stem_3x3s2", 299, 299, 3, 32, 3, 3, 2),
        ConvLayer("stem_3x3", 149, 149, 32, 32, 3, 3),
        ConvLayer("stem_3x3p", 147, 147, 32, 64, 3, 3, 1, (1, 1, 1, 1)),
        ConvLayer("stem_1x1", 73, 73, 64, 80, 1, 1),
        ConvLayer("stem_3x3b", 73, 73, 80, 192, 3, 3),
    ]

    def mixed5(tag, cin, pool_c):
        tot = 64 + 64 + 96 + pool_c
        g = f"mixed{tag}"
        return [
            ConvLayer(f"{g}_b1_1x1", 35, 35, cin, 64, 1, 1, concat=(g, 0, tot)),
            ConvLayer(f"{g}_b2_1x1", 35, 35, cin, 48, 1, 1),
            ConvLayer(f"{g}_b2_5x5", 35, 35, 48, 64, 5, 5, 1, _same(5), concat=(g, 64, tot)),
            ConvLayer(f"{g}_b3_1x1", 35, 35, cin, 64, 1, 1),
            ConvLayer(f"{g}_b3_3x3a", 35, 35, 64, 96, 3, 3, 1, _same(3)),
            ConvLayer(f"{g}_b3_3x3b", 35, 35, 96, 96, 3, 3, 1, _same(3), concat=(g, 128, tot)),
            ConvLayer(f"{g}_b4_1x1", 35, 35, cin, pool_c, 1, 1, concat=(g, 224, tot)),
        ]

    L += mixed5("5b", 192, 32) + mixed5("5c", 256, 64) + mixed5("5d", 288, 64)
    g = "mixed6a"
    L += [
        ConvLayer(f"{g}_b1_3x3s2", 35, 35, 288, 384, 3, 3, 2, concat=(g, 0, 768)),
        ConvLayer(f"{g}_b2_1x1", 35, 35, 288, 64, 1, 1),
        ConvLayer(f"{g}_b2_3x3", 35, 35, 64, 96, 3, 3, 1, _same(3)),
        ConvLayer(f"{g}_b2_3x3s2", 35, 35, 96, 96, 3, 3, 2, concat=(g, 384, 768)),
    ]

    def mixed6(tag, c7):
        g = f"mixed{tag}"
        p17 = (0, 3, 0, 3)  # 1x7: pad width by 3
        p71 = (3, 0, 3, 0)  # 7x1: pad height by 3
        return [
            ConvLayer(f"{g}_b1_1x1", 17, 17, 768, 192, 1, 1, concat=(g, 0, 768)),
            ConvLayer(f"{g}_b2_1x1", 17, 17, 768, c7, 1, 1),
            ConvLayer(f"{g}_b2_1x7", 17, 17, c7, c7, 1, 7, 1, p17),
            ConvLayer(f"{g}_b2_7x1", 17, 17, c7, 192, 7, 1, 1, p71, concat=(g, 192, 768)),
            ConvLayer(f"{g}_b3_1x1", 17, 17, 768, c7, 1, 1),
            ConvLayer(f"{g}_b3_7x1a", 17, 17, c7, c7, 7, 1, 1, p71),
            ConvLayer(f"{g}_b3_1x7a", 17, 17, c7, c7, 1, 7, 1, p17),
            ConvLayer(f"{g}_b3_7x1b", 17, 17, c7, c7, 7, 1, 1, p71),
            ConvLayer(f"{g}_b3_1x7b", 17, 17, c7, 192, 1, 7, 1, p17, concat=(g, 384, 768)),
            ConvLayer(f"{g}_b4_1x1", 17, 17, 768, 192, 1, 1, concat=(g, 576, 768)),
        ]

    for tag, c7 in (("6b", 128), ("6c", 160), ("6d", 160), ("6e", 192)):
        L += mixed6(tag, c7)
    g = "mixed7a"
    L += [
        ConvLayer(f"{g}_b1_1x1", 17, 17, 768, 192, 1, 1),
        ConvLayer(f"{g}_b1_3x3s2", 17, 17, 192, 320, 3, 3, 2, concat=(g, 0, 1280)),
        ConvLayer(f"{g}_b2_1x1", 17, 17, 768, 192, 1, 1),
        ConvLayer(f"{g}_b2_1x7", 17, 17, 192, 192, 1, 7, 1, (0, 3, 0, 3)),
        ConvLayer(f"{g}_b2_7x1", 17, 17, 192, 192, 7, 1, 1, (3, 0, 3, 0)),
        ConvLayer(f"{g}_b2_3x3s2", 17, 17, 192, 192, 3, 3, 2, concat=(g, 320, 1280)),
    ]

    def mixed7(tag, cin):
        g = f"mixed{tag}"
        p13 = (0, 1, 0, 1)
        p31 = (1, 0, 1, 0)
        return [
            ConvLayer(f"{g}_b1_1x1", 8, 8, cin, 320, 1, 1, concat=(g, 0, 2048)),
            ConvLayer(f"{g}_b2_1x1", 8, 8, cin, 384, 1, 1),
            ConvLayer(f"{g}_b2_1x3", 8, 8, 384, 384, 1, 3, 1, p13, concat=(g, 320, 2048)),
            ConvLayer(f"{g}_b2_3x1", 8, 8, 384, 384, 3, 1, 1, p31, concat=(g, 704, 2048)),
            ConvLayer(f"{g}_b3_1x1", 8, 8, cin, 448, 1, 1),
            ConvLayer(f"{g}_b3_3x3", 8, 8, 448, 384, 3, 3, 1, _same(3)),
            ConvLayer(f"{g}_b3_1x3", 8, 8, 384, 384, 1, 3, 1, p13, concat=(g, 1088, 2048)),
            ConvLayer(f"{g}_b3_3x1", 8, 8, 384, 384, 3, 1, 1, p31, concat=(g, 1472, 2048)),
            ConvLayer(f"{g}_b4_1x1", 8, 8, cin, 192, 1, 1, concat=(g, 1856, 2048)),
        ]

    L += mixed7("7b", 1280) + mixed7("7c", 2048)
    return L


# ---------------------------------------------------------------- BERT-base FFN
def bert_ffn(M: int = 128) -> List[DenseLayer]:
    """The two FFN matmuls of a BERT-base layer at M tokens."""
    return [DenseLayer("ffn_up", M, 768, 3072), DenseLayer("ffn_down", M, 3072, 768)]


# The single-layer parity case: 14x14x64 3x3 stride 1 pad 1 at batch 1.
SINGLE_CONV = ConvLayer("conv14x14x64", 14, 14, 64, 64, 3, 3, 1, (1, 1, 1, 1), act=None)
