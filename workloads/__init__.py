"""Seeded synthetic inputs for the batch-1 conv2d workloads.

This module is shared by the CPU oracle's tests and by the GPU path's tests and
benchmark.  It only draws numbers and names shapes: it holds none of the
convolution's arithmetic.

Generator: SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom
number generators", OOPSLA 2014), in its counter form: the i-th output
(i = 1, 2, ...) mixes ``seed + i * 0x9E3779B97F4A7C15``.  A uniform double is
``(z >> 11) * 2**-53``; normals come from the Box-Muller transform with
``u1 = 1 - u`` (so the log never sees 0) and both outputs of each pair used in
order.  Values are produced in float64 and rounded once to float32
(round-to-nearest-even).

The workloads stand in for the paper's ResNet-on-ImageNet layers (Section 5,
Table 2): dense NCHW activations (post-ReLU-like uniform[0,1] except the tiny
case) and He-normal OIHW weights.  Timing does not depend on the values.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def splitmix64(seed: int, n: int) -> np.ndarray:
    """The first ``n`` SplitMix64 outputs for ``seed`` as uint64."""
    i = np.arange(1, n + 1, dtype=np.uint64)
    z = np.uint64(seed & 0xFFFFFFFFFFFFFFFF) + i * _GOLDEN
    z = (z ^ (z >> np.uint64(30))) * _M1
    z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def unit_uniform(seed: int, n: int) -> np.ndarray:
    """n doubles in [0, 1): the top 53 bits of each SplitMix64 output."""
    return (splitmix64(seed, n) >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


def uniform(seed: int, shape, lo: float, hi: float) -> np.ndarray:
    n = int(np.prod(shape))
    u = unit_uniform(seed, n)
    return (lo + (hi - lo) * u).astype(np.float32).reshape(shape)


def normal(seed: int, shape, mean: float, std: float) -> np.ndarray:
    n = int(np.prod(shape))
    pairs = (n + 1) // 2
    u = unit_uniform(seed, 2 * pairs)
    u1 = 1.0 - u[0::2]
    u2 = u[1::2]
    r = np.sqrt(-2.0 * np.log(u1))
    z = np.empty(2 * pairs, dtype=np.float64)
    z[0::2] = r * np.cos(2.0 * math.pi * u2)
    z[1::2] = r * np.sin(2.0 * math.pi * u2)
    return (mean + std * z[:n]).astype(np.float32).reshape(shape)


def small_ints(seed: int, shape, lo: int = -2, hi: int = 2) -> np.ndarray:
    """Integers in [lo, hi] as float32: every partial sum of a conv over them is
    exact in fp32 while it stays below 2**24."""
    n = int(np.prod(shape))
    u = unit_uniform(seed, n)
    v = np.floor(u * (hi - lo + 1)) + lo
    return v.astype(np.float32).reshape(shape)


def he_std(c_in: int, k: int) -> float:
    """He initialisation: standard deviation sqrt(2 / fan_in), fan_in = C_in*K*K."""
    return math.sqrt(2.0 / (c_in * k * k))


@dataclasses.dataclass(frozen=True)
class ConvCase:
    """One batch-1 conv layer: shapes, hyper-parameters and how its tensors are drawn."""
    name: str
    c_in: int
    h: int
    w: int
    c_out: int
    k: int
    stride: int
    pad: int
    x_seed: int
    w_seed: int
    x_dist: tuple          # ("uniform", lo, hi)
    w_dist: tuple          # ("uniform", lo, hi) or ("normal", mean, std)
    bias: str = "none"     # "none" | "zeros" | "normal"
    b_seed: int = 0
    b_std: float = 0.0

    def inputs(self):
        """(x [1,C_in,H,W], w [C_out,C_in,K,K], bias [C_out] or None), float32."""
        x = _draw(self.x_seed, (1, self.c_in, self.h, self.w), self.x_dist)
        wt = _draw(self.w_seed, (self.c_out, self.c_in, self.k, self.k), self.w_dist)
        if self.bias == "none":
            b = None
        elif self.bias == "zeros":
            b = np.zeros(self.c_out, dtype=np.float32)
        else:
            b = normal(self.b_seed, (self.c_out,), 0.0, self.b_std)
        return x, wt, b

    def dims(self):
        return dict(c_in=self.c_in, h=self.h, w=self.w, c_out=self.c_out,
                    k=self.k, stride=self.stride, pad=self.pad)


def _draw(seed, shape, dist):
    if dist[0] == "uniform":
        return uniform(seed, shape, dist[1], dist[2])
    if dist[0] == "normal":
        return normal(seed, shape, dist[1], dist[2])
    raise ValueError(dist)


def _he(c_in, k):
    return ("normal", 0.0, he_std(c_in, k))


# The five workloads.  Readings where the workload text is silent:
#  * the 1x1 layer on 7x7 uses pad 0 (only the 5x5 layer names pad 2);
#  * layers whose bias is not named take no bias (NULL), the tiny case passes an
#    explicit zero buffer;
#  * normal(0, s) takes s as the standard deviation; the strided layer uses its
#    own fan-in (128*9).
TINY = ConvCase("tiny_3to16_32x32", 3, 32, 32, 16, 3, 1, 1, 1001, 1002,
                ("uniform", -1.0, 1.0), ("uniform", -0.5, 0.5), bias="zeros")
VGG_EARLY = ConvCase("vgg_early_64to64_224x224", 64, 224, 224, 64, 3, 1, 1, 2001, 2002,
                     ("uniform", 0.0, 1.0), _he(64, 3), bias="normal", b_seed=2003, b_std=0.01)
RESNET_CONV4 = ConvCase("resnet_conv4_256to256_14x14", 256, 14, 14, 256, 3, 1, 1, 3001, 3002,
                        ("uniform", 0.0, 1.0), _he(256, 3))
RESNET_STRIDED = ConvCase("resnet_strided_128to256_28x28_s2", 128, 28, 28, 256, 3, 2, 1, 3101, 3102,
                          ("uniform", 0.0, 1.0), _he(128, 3))
DEEP_1X1 = ConvCase("deep_1x1_512to512_7x7", 512, 7, 7, 512, 1, 1, 0, 4001, 4002,
                    ("uniform", 0.0, 1.0), _he(512, 1))
DEEP_5X5 = ConvCase("deep_5x5_512to512_7x7", 512, 7, 7, 512, 5, 1, 2, 4001, 4003,
                    ("uniform", 0.0, 1.0), _he(512, 5))

SINGLE_LAYER_CASES = [TINY, VGG_EARLY, RESNET_CONV4, RESNET_STRIDED, DEEP_1X1, DEEP_5X5]

# The other 3x3 layers of ResNet's Table 2 set (conv2.x, conv3.x, conv5.x; conv4.x is
# RESNET_CONV4), batch 1, post-ReLU-like inputs and He-normal weights, no bias.
RESNET_CONV2 = ConvCase("resnet_conv2_64to64_56x56", 64, 56, 56, 64, 3, 1, 1, 3201, 3202,
                        ("uniform", 0.0, 1.0), _he(64, 3))
RESNET_CONV3 = ConvCase("resnet_conv3_128to128_28x28", 128, 28, 28, 128, 3, 1, 1, 3301, 3302,
                        ("uniform", 0.0, 1.0), _he(128, 3))
RESNET_CONV5 = ConvCase("resnet_conv5_512to512_7x7", 512, 7, 7, 512, 3, 1, 1, 3501, 3502,
                        ("uniform", 0.0, 1.0), _he(512, 3))
RESNET_3X3_CASES = [RESNET_CONV2, RESNET_CONV3, RESNET_CONV4, RESNET_CONV5]

# The first VGG-16 layer on its own (3 input channels: the memory-bound case).
VGG16_CONV1_1 = ConvCase("vgg16_conv1_1_3to64_224x224", 3, 224, 224, 64, 3, 1, 1, 5001, 5100,
                         ("uniform", 0.0, 1.0), _he(3, 3))

EXTRA_CASES = [RESNET_CONV2, RESNET_CONV3, RESNET_CONV5, VGG16_CONV1_1]
ALL_CASES = SINGLE_LAYER_CASES + EXTRA_CASES

# Batch-1 VGG-16 conv stack: 13 3x3/pad-1/stride-1 convs, ReLU after each,
# 2x2/stride-2 max-pool after stages 1-4 (none after stage 5).
VGG16_STAGES = [[(3, 64), (64, 64)],
                [(64, 128), (128, 128)],
                [(128, 256), (256, 256), (256, 256)],
                [(256, 512), (512, 512), (512, 512)],
                [(512, 512), (512, 512), (512, 512)]]
VGG16_INPUT_SEED = 5001
VGG16_HW = 224


def vgg16_layers():
    """[(name, C_in, C_out, H, pool_after, weight_seed)] for the 13 convs."""
    out = []
    hw = VGG16_HW
    idx = 0
    for si, stage in enumerate(VGG16_STAGES):
        for li, (ci, co) in enumerate(stage):
            idx += 1
            pool = (li == len(stage) - 1) and si < len(VGG16_STAGES) - 1
            out.append((f"conv{si + 1}_{li + 1}", ci, co, hw, pool, 5100 + idx))
        hw //= 2
    return out


def vgg16_input() -> np.ndarray:
    return uniform(VGG16_INPUT_SEED, (1, 3, VGG16_HW, VGG16_HW), 0.0, 1.0)


def vgg16_weights(ci: int, co: int, seed: int) -> np.ndarray:
    return normal(seed, (co, ci, 3, 3), 0.0, he_std(ci, 3))


def fuzz_shapes(seed: int, n: int):
    """Random small conv shapes (C_in 1-17, C_out 1-70, H,W 1-23, K in {1,2,3,4,5,7},
    stride 1-3, pad 0..K), keeping only those with at least one output pixel."""
    u = unit_uniform(seed, 16 * n * 8)
    j = 0
    shapes = []
    ks = [1, 2, 3, 4, 5, 7]

    def pick(lo, hi):
        nonlocal j
        v = lo + int(u[j] * (hi - lo + 1))
        j += 1
        return min(v, hi)

    while len(shapes) < n and j + 8 <= len(u):
        c_in, c_out = pick(1, 17), pick(1, 70)
        h, w = pick(1, 23), pick(1, 23)
        k = ks[pick(0, 5)]
        s = pick(1, 3)
        p = pick(0, k)
        if (h + 2 * p - k) < 0 or (w + 2 * p - k) < 0:
            continue
        shapes.append(dict(c_in=c_in, h=h, w=w, c_out=c_out, k=k, stride=s, pad=p))
    return shapes


def to_device(torch, a):
    """A contiguous float32 CUDA copy of a host array (None stays None)."""
    if a is None:
        return None
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def case_by_name(name: str) -> Optional[ConvCase]:
    for c in ALL_CASES:
        if c.name == name:
            return c
    return None
