"""Seeded synthetic inputs and the conv layer tables of the evaluated networks.

This module is shared by the product side (bench, binding tests) and by the
tests of the CPU oracle, so it holds no arithmetic of the convolution itself:
only layer shapes written out as literals, seeds, and random draws.

Networks (Sec. 4.1 evaluates GluonCV ResNet50_v1 and MobileNet1.0 at batch 1;
VGG-16 is an extra compute-dense stack).  Every layer lists its input extent
explicitly so that nothing here derives an output size.

Seeds: ``190702154 + 1000*config + 10*layer + t`` with t = 0 for the input,
1 for the weights, 2 for the bias, drawn with a CPU ``torch.Generator``.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np
import torch

SEED_BASE = 190702154


@dataclass(frozen=True)
class ConvLayer:
    name: str
    N: int
    C: int
    H: int
    W: int
    K: int
    R: int
    S: int
    stride: int
    pad: int
    groups: int = 1
    relu: bool = True
    # kind: "dense" (conv2d_fwd) or "dw" (dwconv2d_fwd)
    kind: str = "dense"
    # distribution of this layer's input when it is drawn on its own:
    # "u01" = uniform[0,1), "n01" = standard normal
    xdist: str = "u01"

    @property
    def fan_in(self) -> int:
        return (self.C // self.groups) * self.R * self.S

    @property
    def he_std(self) -> float:
        return math.sqrt(2.0 / self.fan_in)

    def with_batch(self, N: int) -> "ConvLayer":
        return ConvLayer(self.name, N, self.C, self.H, self.W, self.K, self.R, self.S,
                         self.stride, self.pad, self.groups, self.relu, self.kind, self.xdist)


@dataclass
class Workload:
    config: int
    name: str
    layers: List[ConvLayer]
    dtype: str = "f32"          # "f32" or "bf16" (x and w in bf16, fp32 accumulate/output)
    notes: str = ""
    extra: dict = field(default_factory=dict)


def _resnet50_v1(N: int, xdist: str = "u01") -> List[ConvLayer]:
    """ResNet-50 v1 (GluonCV ResNet50_v1): 7x7/2 stem, bottlenecks [3,4,6,3],
    widths 64/128/256/512, expansion 4; the stride-2 of stages 3-5 sits on the
    first 1x1 of the first block, as does the 1x1 projection shortcut."""
    L = [ConvLayer("stem", N, 3, 224, 224, 64, 7, 7, 2, 3, relu=True, xdist=xdist)]
    # (stage name, blocks, width, input channels, input extent, first stride)
    stages = [("s2", 3, 64, 64, 56, 1),
              ("s3", 4, 128, 256, 56, 2),
              ("s4", 6, 256, 512, 28, 2),
              ("s5", 3, 512, 1024, 14, 2)]
    out_extent = {"s2": 56, "s3": 28, "s4": 14, "s5": 7}
    for sname, blocks, width, cin, ext_in, st in stages:
        e = out_extent[sname]
        for b in range(blocks):
            c_in = cin if b == 0 else 4 * width
            h_in = ext_in if b == 0 else e
            s1 = st if b == 0 else 1
            L.append(ConvLayer(f"{sname}b{b}c1", N, c_in, h_in, h_in, width, 1, 1, s1, 0, relu=True))
            L.append(ConvLayer(f"{sname}b{b}c2", N, width, e, e, width, 3, 3, 1, 1, relu=True))
            L.append(ConvLayer(f"{sname}b{b}c3", N, width, e, e, 4 * width, 1, 1, 1, 0, relu=False))
            if b == 0:
                L.append(ConvLayer(f"{sname}b{b}proj", N, c_in, h_in, h_in, 4 * width, 1, 1, s1, 0,
                                   relu=False))
    return L


def _mobilenet_v1(N: int) -> List[ConvLayer]:
    """MobileNet-v1 1.0: 3x3/2 stem to 32 channels, then 13 (dw 3x3 pad 1,
    pw 1x1) pairs; bias + ReLU after every conv."""
    L = [ConvLayer("stem", N, 3, 224, 224, 32, 3, 3, 2, 1, relu=True)]
    # (dw channels, dw input extent, dw stride, dw output extent, pw output channels)
    pairs = [(32, 112, 1, 112, 64), (64, 112, 2, 56, 128), (128, 56, 1, 56, 128),
             (128, 56, 2, 28, 256), (256, 28, 1, 28, 256), (256, 28, 2, 14, 512),
             (512, 14, 1, 14, 512), (512, 14, 1, 14, 512), (512, 14, 1, 14, 512),
             (512, 14, 1, 14, 512), (512, 14, 1, 14, 512), (512, 14, 2, 7, 1024),
             (1024, 7, 1, 7, 1024)]
    for i, (c, hin, st, hout, k) in enumerate(pairs, start=1):
        L.append(ConvLayer(f"dw{i}", N, c, hin, hin, c, 3, 3, st, 1, groups=c, relu=True, kind="dw"))
        L.append(ConvLayer(f"pw{i}", N, c, hout, hout, k, 1, 1, 1, 0, relu=True))
    return L


def _vgg16(N: int) -> List[ConvLayer]:
    """VGG-16 conv stack: 13 3x3/1 pad-1 convs in 5 stages (64,128,256,512,512),
    a 2x2/2 max-pool between stages."""
    spec = [(224, [(3, 64), (64, 64)]),
            (112, [(64, 128), (128, 128)]),
            (56, [(128, 256), (256, 256), (256, 256)]),
            (28, [(256, 512), (512, 512), (512, 512)]),
            (14, [(512, 512), (512, 512), (512, 512)])]
    L = []
    for si, (ext, convs) in enumerate(spec, start=1):
        for ci, (c, k) in enumerate(convs, start=1):
            L.append(ConvLayer(f"conv{si}_{ci}", N, c, ext, ext, k, 3, 3, 1, 1, relu=True,
                               xdist="n01" if (si, ci) == (1, 1) else "u01"))
    return L


def _squeezenet10(N: int) -> List[ConvLayer]:
    """SqueezeNet 1.0 (Iandola et al., 2016; the third classification model of
    Sec. 4.1): 7x7/2 stem to 96 channels (no padding, 224 -> 109), 3x3/2
    max-pools (ceil mode: 109 -> 54 -> 27 -> 13) before fire2, fire5 and
    fire9, eight fire modules, each a 1x1 squeeze conv followed by a 1x1 and a
    3x3 (pad 1) expand conv whose outputs are concatenated along channels
    (expand1x1 first), and a 1x1 classifier conv to 1000 channels; bias +
    ReLU after every conv."""
    L = [ConvLayer("conv1", N, 3, 224, 224, 96, 7, 7, 2, 0, relu=True)]
    # (fire index, input channels, squeeze, expand per branch, extent)
    fires = [(2, 96, 16, 64, 54), (3, 128, 16, 64, 54), (4, 128, 32, 128, 54),
             (5, 256, 32, 128, 27), (6, 256, 48, 192, 27), (7, 384, 48, 192, 27),
             (8, 384, 64, 256, 27), (9, 512, 64, 256, 13)]
    for f, cin, sq, ex, e in fires:
        L.append(ConvLayer(f"fire{f}_squeeze", N, cin, e, e, sq, 1, 1, 1, 0, relu=True))
        L.append(ConvLayer(f"fire{f}_expand1x1", N, sq, e, e, ex, 1, 1, 1, 0, relu=True))
        L.append(ConvLayer(f"fire{f}_expand3x3", N, sq, e, e, ex, 3, 3, 1, 1, relu=True))
    L.append(ConvLayer("conv10", N, 512, 13, 13, 1000, 1, 1, 1, 0, relu=True))
    return L


def workload(config: int, batch: Optional[int] = None) -> Workload:
    """The five evaluation configurations (1-based), and 6: SqueezeNet 1.0 at
    batch 1 (the paper's third model)."""
    if config == 1:
        L = [ConvLayer("conv3x3_64", 1, 64, 56, 56, 64, 3, 3, 1, 1, relu=True)]
        w = Workload(1, "conv3x3 64->64 @56x56 b1 fp32", L)
    elif config == 2:
        w = Workload(2, "ResNet-50 v1 conv stack b1 fp32", _resnet50_v1(1))
    elif config == 3:
        w = Workload(3, "MobileNet-v1 1.0 conv stack b1 fp32", _mobilenet_v1(1))
    elif config == 4:
        w = Workload(4, "VGG-16 conv stack b8 fp32", _vgg16(8))
    elif config == 5:
        w = Workload(5, "ResNet-50 v1 conv stack b64 bf16-in fp32-acc", _resnet50_v1(64), dtype="bf16")
    elif config == 6:
        w = Workload(6, "SqueezeNet 1.0 conv stack b1 fp32", _squeezenet10(1))
    else:
        raise ValueError(f"no config {config}")
    if batch is not None:
        w.layers = [l.with_batch(batch) for l in w.layers]
        w.name = w.name + f" (batch {batch})"
    return w


def seed(config: int, layer: int, t: int) -> int:
    return SEED_BASE + 1000 * config + 10 * layer + t


def _gen(s: int) -> torch.Generator:
    g = torch.Generator(device="cpu")
    g.manual_seed(s)
    return g


def uniform01(shape, s: int) -> np.ndarray:
    return torch.rand(tuple(shape), generator=_gen(s), dtype=torch.float32).numpy()


def normal(shape, std: float, s: int) -> np.ndarray:
    return (torch.randn(tuple(shape), generator=_gen(s), dtype=torch.float32) * std).numpy()


def small_ints(shape, lo: int, hi: int, s: int) -> np.ndarray:
    """Integers in [lo, hi] stored as fp32: exact in fp32 and bf16, so any
    summation order gives the same result while partial sums stay below 2^24."""
    return torch.randint(lo, hi + 1, tuple(shape), generator=_gen(s)).to(torch.float32).numpy()


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round to nearest even, torch's cast) and return the bit patterns."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def layer_tensors(config: int, index: int, layer: ConvLayer):
    """Seeded host tensors (x, w, bias) for one layer drawn on its own:
    x per the layer's distribution, w He-normal std sqrt(2/fan_in),
    bias N(0, 0.01).  Shapes: x [N][C][H][W], w [K][C/groups][R][S], bias [K]."""
    xs = (layer.N, layer.C, layer.H, layer.W)
    ws = (layer.K, layer.C // layer.groups, layer.R, layer.S)
    if layer.xdist == "n01":
        x = normal(xs, 1.0, seed(config, index, 0))
    else:
        x = uniform01(xs, seed(config, index, 0))
    w = normal(ws, layer.he_std, seed(config, index, 1))
    b = normal((layer.K,), 0.01, seed(config, index, 2))
    return x, w, b


def flops(layer: ConvLayer, P: int, Q: int) -> int:
    """Multiply-adds counted as 2 FLOP: 2*N*K*P*Q*(C/groups)*R*S (epilogue not counted)."""
    return 2 * layer.N * layer.K * P * Q * (layer.C // layer.groups) * layer.R * layer.S
