"""Synthetic layer workloads: shapes and seeded FP32 input generators.

Holds none of the method's arithmetic -- only layer shapes and random FP32
tensors -- so that the HIP path (tests, benchmark) and the CPU oracle can be
fed identical inputs.  The paper trains on ImageNet-1K (Sec. 5), which is not
available here; per-layer Gaussian tensors at the paper's network shapes stand
in for it:
  * activations: N(0,1), or ReLU(N(0,1)) for post-activation feature maps,
  * weights: He-normal N(0, 2 / (C*R*S)),
  * output gradients: N(0,1) or N(0,1) * 1e-3.
Each layer draws from ``np.random.default_rng((config_seed, layer_index))``
with ``standard_normal(dtype=float32)``, in the order x, w, dy.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np


@dataclasses.dataclass(frozen=True)
class Layer:
    name: str
    n: int
    c: int
    h: int
    w: int
    k: int
    r: int
    s: int
    stride: int = 1
    pad: int = 0

    @property
    def p(self) -> int:
        return (self.h + 2 * self.pad - self.r) // self.stride + 1

    @property
    def q(self) -> int:
        return (self.w + 2 * self.pad - self.s) // self.stride + 1

    @property
    def macs(self) -> int:
        """Multiply-accumulates of one direction (the same for all three)."""
        return self.n * self.k * self.c * self.r * self.s * self.p * self.q

    def shapes(self):
        return ((self.n, self.c, self.h, self.w), (self.k, self.c, self.r, self.s),
                (self.n, self.k, self.p, self.q))


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    layers: List[Layer]
    seed: int
    x_dist: str          # "normal" | "relu"
    dy_scale: float
    roundings: tuple
    chunk_lens: tuple
    w_scale: Optional[float] = None  # None -> He-normal sqrt(2 / (C*R*S))


def resnet50_v1_convs(n: int = 64) -> List[Layer]:
    """The 53 convolutions of ResNet-50 v1 (stride on the first 1x1 of stages
    3-5 and on the projection shortcuts) at 224x224 input."""
    layers = [Layer("conv1", n, 3, 224, 224, 64, 7, 7, 2, 3)]
    h = 56
    cin = 64
    for stage, (blocks, mid, out) in enumerate(((3, 64, 256), (4, 128, 512), (6, 256, 1024), (3, 512, 2048)), 2):
        for b in range(blocks):
            stride = 2 if (b == 0 and stage > 2) else 1
            ho = h // stride
            tag = "res%d%s" % (stage, "abcdef"[b])
            layers.append(Layer(tag + "_branch2a", n, cin, h, h, mid, 1, 1, stride, 0))
            layers.append(Layer(tag + "_branch2b", n, mid, ho, ho, mid, 3, 3, 1, 1))
            layers.append(Layer(tag + "_branch2c", n, mid, ho, ho, out, 1, 1, 1, 0))
            if b == 0:
                layers.append(Layer(tag + "_branch1", n, cin, h, h, out, 1, 1, stride, 0))
            cin = out
            h = ho
    return layers


WORKLOADS = {
    # Single layer: N=2, C=16, 14x14, K=32, 3x3 s1 p1; x, dy ~ N(0,1);
    # w ~ N(0,1) * sqrt(2/(C*9)); seed 0; nearest; L = 16.
    "layer16x32": Workload("layer16x32", [Layer("layer16x32", 2, 16, 14, 14, 32, 3, 3, 1, 1)], 0, "normal", 1.0,
                           ("nearest",), (16,)),
    # ResNet-50 conv2_x 3x3: N=32, 64->64 at 56x56; ReLU(N(0,1)) activations,
    # He weights, dy ~ N(0,1e-3); stochastic, seed 1; L in {8,16,32,64}.
    "resnet50_conv2x_3x3": Workload("resnet50_conv2x_3x3", [Layer("res2_3x3", 32, 64, 56, 56, 64, 3, 3, 1, 1)], 1,
                                    "relu", 1e-3, ("stochastic",), (8, 16, 32, 64)),
    # ResNet-50 conv4_x 1x1 bottleneck pair at N=64, 14x14.
    "resnet50_conv4x_1x1": Workload("resnet50_conv4x_1x1",
                                    [Layer("res4_1x1_1024to256", 64, 1024, 14, 14, 256, 1, 1),
                                     Layer("res4_1x1_256to1024", 64, 256, 14, 14, 1024, 1, 1)], 3,
                                    "relu", 1e-3, ("nearest", "biased"), (64,)),
    # VGG-16 conv1_2 (64->64 at 224) and conv3_3 (256->256 at 56), N=32.
    "vgg16_conv1_2_conv3_3": Workload("vgg16_conv1_2_conv3_3",
                                      [Layer("vgg_conv1_2", 32, 64, 224, 224, 64, 3, 3, 1, 1),
                                       Layer("vgg_conv3_3", 32, 256, 56, 56, 256, 3, 3, 1, 1)], 2,
                                      "relu", 1e-3, ("stochastic",), (64,)),
    # All 53 ResNet-50 v1 convolutions at N=64, x ~ N(0,1), dy ~ N(0,1).
    "resnet50_all_convs": Workload("resnet50_all_convs", resnet50_v1_convs(64), 5, "normal", 1.0,
                                   ("nearest",), (64,)),
}


def layer_inputs(wl: Workload, index: int, scale_n: Optional[int] = None):
    """FP32 (x, w, dy) of layer `index` of a workload, generated on the host.

    scale_n (optional) replaces the batch size, for reduced-size test cases."""
    layer = wl.layers[index]
    if scale_n is not None:
        layer = dataclasses.replace(layer, n=scale_n)
    rng = np.random.default_rng((wl.seed, index))
    xs, ws, ds = layer.shapes()
    x = rng.standard_normal(xs, dtype=np.float32)
    w = rng.standard_normal(ws, dtype=np.float32)
    dy = rng.standard_normal(ds, dtype=np.float32)
    if wl.x_dist == "relu":
        np.maximum(x, 0, out=x)
    wsc = wl.w_scale if wl.w_scale is not None else float(np.sqrt(2.0 / (layer.c * layer.r * layer.s)))
    w *= np.float32(wsc)
    if wl.dy_scale != 1.0:
        dy *= np.float32(wl.dy_scale)
    return layer, x, w, dy
