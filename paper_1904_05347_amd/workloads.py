"""Seeded synthetic inputs and the workload table.

This module holds no arithmetic of the method: it only names the problem
shapes (the paper's VGG-16 and ResNet-50 layer tables of Section 5 and its
power-of-two GEMM sweep, here at batch 32 and at 4096^3) and draws their
inputs.  Both the HIP path's tests/benchmark and the CPU oracle receive the
very same host arrays from here.

Values are i.i.d. uniform on [-1, 1): numpy PCG64 ``random(n, float32)`` is a
multiple of 2**-24 in [0, 1), so ``2*u - 1`` is exact in fp32 and lies on a
2**-23 grid.  Products of two such values are multiples of 2**-46 or exactly 0,
so no denormal can arise.  Integer-valued inputs (every partial sum exact in
fp32) come from ``integers``.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


def uniform(rng: np.random.Generator, n: int) -> np.ndarray:
    """n fp32 values, i.i.d. uniform on a 2**-23 grid in [-1, 1)."""
    u = rng.random(n, dtype=np.float32)
    return u * np.float32(2.0) - np.float32(1.0)


def integers(rng: np.random.Generator, n: int, lo: int = -8, hi: int = 8) -> np.ndarray:
    """n fp32 values, i.i.d. uniform integers in [lo, hi]."""
    return rng.integers(lo, hi + 1, size=n).astype(np.float32)


def _draw(rng, n, kind):
    if kind == "uniform":
        return uniform(rng, n)
    if kind == "int":
        return integers(rng, n)
    raise ValueError(kind)


# ------------------------------------------------------------------ GEMM

@dataclass(frozen=True)
class GemmCase:
    """C = alpha op(A) op(B) + beta C, row-major, contiguous storage."""
    name: str
    trans_a: str
    trans_b: str
    M: int
    N: int
    K: int
    alpha: float
    beta: float
    seed: int

    @property
    def a_shape(self):
        return (self.K, self.M) if self.trans_a == "T" else (self.M, self.K)

    @property
    def b_shape(self):
        return (self.N, self.K) if self.trans_b == "T" else (self.K, self.N)

    @property
    def lda(self):
        return self.a_shape[1]

    @property
    def ldb(self):
        return self.b_shape[1]

    @property
    def ldc(self):
        return self.N

    @property
    def flops(self):
        return 2 * self.M * self.N * self.K

    def inputs(self, kind: str = "uniform"):
        """(A, B, C) as 2-D float32 arrays in storage shape; C is drawn only when beta != 0."""
        rng = np.random.default_rng(self.seed)
        A = _draw(rng, self.a_shape[0] * self.a_shape[1], kind).reshape(self.a_shape)
        B = _draw(rng, self.b_shape[0] * self.b_shape[1], kind).reshape(self.b_shape)
        if self.beta != 0.0:
            C = _draw(rng, self.M * self.N, kind).reshape(self.M, self.N)
        else:
            C = np.zeros((self.M, self.N), dtype=np.float32)
        return A, B, C


# ----------------------------------------------------------- convolution

@dataclass(frozen=True)
class ConvCase:
    """NHWC input, HWIO filter, explicit padding (top, left, bottom, right)."""
    name: str
    N: int
    H: int
    W: int
    Cin: int
    KH: int
    KW: int
    Cout: int
    stride: tuple = (1, 1)
    pads: tuple = (0, 0, 0, 0)
    seed: int = 0
    # Output size stated by the source table (checked, never used as input).
    out_hw: tuple = field(default=None)

    @property
    def x_shape(self):
        return (self.N, self.H, self.W, self.Cin)

    @property
    def f_shape(self):
        return (self.KH, self.KW, self.Cin, self.Cout)

    def inputs(self, kind: str = "uniform"):
        """(x, f) as float32 arrays, NHWC and HWIO."""
        rng = np.random.default_rng(self.seed)
        x = _draw(rng, int(np.prod(self.x_shape)), kind).reshape(self.x_shape)
        f = _draw(rng, int(np.prod(self.f_shape)), kind).reshape(self.f_shape)
        return x, f


def conv_flops(case: ConvCase, Ho: int, Wo: int) -> int:
    """Nominal multiply-adds x 2, padded taps included."""
    return 2 * case.N * Ho * Wo * case.Cout * case.KH * case.KW * case.Cin


# The parity-size problems: small enough for the whole oracle in seconds.
GEMM_SMALL = GemmCase("gemm NN 512x512x512 alpha=1 beta=0", "N", "N", 512, 512, 512, 1.0, 0.0, 1)
CONV_SMALL = ConvCase("conv b1 56x56x64->64 3x3 s1 same", 1, 56, 56, 64, 3, 3, 64,
                      (1, 1), (1, 1, 1, 1), 2, (56, 56))

# The GEMM sweep: square sizes, then the two transposed layouts at 4096.
GEMM_SWEEP = [
    GemmCase("gemm NN 1024^3 beta=0.5", "N", "N", 1024, 1024, 1024, 1.0, 0.5, 31),
    GemmCase("gemm NN 2048^3 beta=0.5", "N", "N", 2048, 2048, 2048, 1.0, 0.5, 32),
    GemmCase("gemm NN 4096^3 beta=0.5", "N", "N", 4096, 4096, 4096, 1.0, 0.5, 33),
    GemmCase("gemm TN 4096^3 beta=0.5", "T", "N", 4096, 4096, 4096, 1.0, 0.5, 34),
    GemmCase("gemm NT 4096^3 beta=0.5", "N", "T", 4096, 4096, 4096, 1.0, 0.5, 35),
]

# VGG-16 first layer of each block (the paper's VGG layer table), batch 32,
# 3x3 stride 1 with one pixel of zero padding on every side ("same").
_S1 = (1, 1)
_P1 = (1, 1, 1, 1)
_P0 = (0, 0, 0, 0)
VGG_LAYERS = [
    ConvCase("vgg16 conv1_1 b32 224x224x3->64 3x3", 32, 224, 224, 3, 3, 3, 64, _S1, _P1, 41, (224, 224)),
    ConvCase("vgg16 conv2_1 b32 112x112x64->128 3x3", 32, 112, 112, 64, 3, 3, 128, _S1, _P1, 42, (112, 112)),
    ConvCase("vgg16 conv3_1 b32 56x56x128->256 3x3", 32, 56, 56, 128, 3, 3, 256, _S1, _P1, 43, (56, 56)),
    ConvCase("vgg16 conv4_1 b32 28x28x256->512 3x3", 32, 28, 28, 256, 3, 3, 512, _S1, _P1, 44, (28, 28)),
    ConvCase("vgg16 conv5_1 b32 14x14x512->512 3x3", 32, 14, 14, 512, 3, 3, 512, _S1, _P1, 45, (14, 14)),
]

# ResNet-50 bottleneck layers, batch 32.  The stride-2 1x1 layer reads a
# 56x56x256 map and writes 28x28x128 (the down-sampling branch of the first
# block of the third stage).
RESNET_LAYERS = [
    ConvCase("resnet50 b32 56x56x64->64 1x1", 32, 56, 56, 64, 1, 1, 64, _S1, _P0, 51, (56, 56)),
    ConvCase("resnet50 b32 56x56x64->64 3x3", 32, 56, 56, 64, 3, 3, 64, _S1, _P1, 52, (56, 56)),
    ConvCase("resnet50 b32 56x56x64->256 1x1", 32, 56, 56, 64, 1, 1, 256, _S1, _P0, 53, (56, 56)),
    ConvCase("resnet50 b32 56x56x256->128 1x1 s2", 32, 56, 56, 256, 1, 1, 128, (2, 2), _P0, 54, (28, 28)),
    ConvCase("resnet50 b32 7x7x2048->512 1x1", 32, 7, 7, 2048, 1, 1, 512, _S1, _P0, 55, (7, 7)),
]

# The other reading of the stride-2 row: the paper's 28x28x512 -> 128 1x1 layer.
RESNET_ALT = ConvCase("resnet50 b32 28x28x512->128 1x1", 32, 28, 28, 512, 1, 1, 128, _S1, _P0, 56, (28, 28))

# The benchmark's step: the three 4096^3 GEMMs and the ten conv layers.
STEP_GEMMS = GEMM_SWEEP[2:]
STEP_CONVS = VGG_LAYERS + RESNET_LAYERS


# ---------------------------------------------------------------- suites
# Every distinct convolution layer of the paper's VGG-16 and ResNet-50
# tables: (name, window, stride, input H (= W), Cin, Cout, pads t/l/b/r).
# The pads are "same" padding written out (3x3 stride 1: one pixel all
# round; 3x3 stride 2: the odd pixel at the bottom/right; 1x1: none) and none
# for the 7x7 stride-2 first ResNet layer, whose 230 x 230 input is the
# 224 x 224 image already padded by 3.
_SAME3 = (1, 1, 1, 1)
_SAME3S2 = (0, 0, 1, 1)
_NONE = (0, 0, 0, 0)
VGG16_TABLE = [
    ("conv1_1", 3, 1, 224, 3, 64, _SAME3), ("conv1_2", 3, 1, 224, 64, 64, _SAME3),
    ("conv2_1", 3, 1, 112, 64, 128, _SAME3), ("conv2_2", 3, 1, 112, 128, 128, _SAME3),
    ("conv3_1", 3, 1, 56, 128, 256, _SAME3), ("conv3_2", 3, 1, 56, 256, 256, _SAME3),
    ("conv4_1", 3, 1, 28, 256, 512, _SAME3), ("conv4_2", 3, 1, 28, 512, 512, _SAME3),
    ("conv5_1", 3, 1, 14, 512, 512, _SAME3),
]
RESNET50_TABLE = [
    ("conv1_1", 7, 2, 230, 3, 64, _NONE),
    ("conv2_1", 1, 1, 56, 64, 256, _NONE), ("conv2_2", 1, 1, 56, 64, 64, _NONE),
    ("conv2_3", 3, 1, 56, 64, 64, _SAME3), ("conv2_4", 1, 1, 56, 256, 64, _NONE),
    ("conv2_5", 3, 2, 56, 64, 64, _SAME3S2),
    ("conv3_1", 1, 1, 28, 64, 256, _NONE), ("conv3_2", 1, 1, 28, 256, 512, _NONE),
    ("conv3_3", 1, 1, 28, 256, 128, _NONE), ("conv3_4", 3, 1, 28, 128, 128, _SAME3),
    ("conv3_5", 1, 1, 28, 128, 512, _NONE), ("conv3_6", 1, 1, 28, 512, 128, _NONE),
    ("conv3_7", 3, 2, 28, 128, 128, _SAME3S2),
    ("conv4_1", 1, 1, 14, 128, 512, _NONE), ("conv4_2", 1, 1, 14, 512, 1024, _NONE),
    ("conv4_3", 1, 1, 14, 512, 256, _NONE), ("conv4_4", 3, 1, 14, 256, 256, _SAME3),
    ("conv4_5", 1, 1, 14, 256, 1024, _NONE), ("conv4_6", 1, 1, 14, 1024, 256, _NONE),
    ("conv4_7", 3, 2, 14, 256, 256, _SAME3S2),
    ("conv5_1", 1, 1, 7, 256, 1024, _NONE), ("conv5_2", 1, 1, 7, 1024, 2048, _NONE),
    ("conv5_3", 1, 1, 7, 1024, 512, _NONE), ("conv5_4", 3, 1, 7, 512, 512, _SAME3),
    ("conv5_5", 1, 1, 7, 512, 2048, _NONE), ("conv5_6", 1, 1, 7, 2048, 512, _NONE),
]


def layer_suite(batch: int):
    """Every distinct layer of both tables at the given batch, as ConvCases."""
    cases = []
    for net, table, seed0 in (("vgg16", VGG16_TABLE, 100), ("resnet50", RESNET50_TABLE, 200)):
        for i, (name, k, s, hw, cin, cout, pads) in enumerate(table):
            cases.append(ConvCase("%s %s b%d %dx%dx%d->%d %dx%d s%d" % (net, name, batch, hw, hw, cin, cout, k, k, s),
                                  batch, hw, hw, cin, k, k, cout, (s, s), pads, seed0 + 1000 * batch + i))
    return cases


# The paper's GEMM sweep: M, N, K each a power of two in [64, 1024].
SWEEP_SIZES = (64, 128, 256, 512, 1024)


def gemm_sweep():
    cases = []
    for M in SWEEP_SIZES:
        for N in SWEEP_SIZES:
            for K in SWEEP_SIZES:
                cases.append(GemmCase("gemm NN %dx%dx%d" % (M, N, K), "N", "N", M, N, K, 1.0, 0.0,
                                      7000 + M + 3 * N + 7 * K))
    return cases
