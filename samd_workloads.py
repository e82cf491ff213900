"""Seeded synthetic inputs for the SAMD quantized-convolution workloads.

This module is shared by the CPU oracle (``oracle/``) and the GPU path's tests and
benchmark.  It draws integers and describes shapes; it holds none of the method's
arithmetic (no packing, no convolution, no requantisation).

Every input is synthetic: no trained weights or images are used.  The paper measures
the convolution layers of VGG-B (Experimental Setup, Sec. 7) with N-bit signed weights
and activations, N = 8 down to 2; workload 6 has those layer shapes (the published
architecture: 3x3 kernels, stride 1, pad 1, batch 1) with uniform synthetic values.
Workloads 1-5 are the other cases:

1. ``single``  - one conv2d layer, 1x16x16x16 -> 16 channels, 3x3, stride 1, pad 1,
   unsigned b-bit activations, signed b-bit weights (b = 4 by default).
2. ``conv1d``  - standalone 1-D convolution of 2**20 unsigned b-bit values with an
   unsigned 3- or 5-tap kernel.
3. ``mid``     - conv2d 8x128x56x56 -> 128, 3x3, stride 1, pad 1, unsigned x signed.
4. ``stress``  - conv2d 4x256x28x28 -> 256, 3x3, pad 1, signed x signed with half of
   the values at the two range extremes (sign fix-up and carry stress).
5. ``alexnet`` - five-layer AlexNet-shaped stack on 16x3x224x224 (11x11/4 96ch,
   5x5 256ch, 3x3 384ch, 3x3 384ch, 3x3 256ch), unsigned activations, signed weights.
6. ``vggb``    - the ten VGG-B convolution layers, each on its own (batch 1, input
   sizes as after VGG-B's max-pools: 224, 224, 112, 112, 56, 56, 28, 28, 14, 14),
   signed b-bit activations and weights, uniform; seed offset = layer index.

Value recipe: numpy ``Generator(PCG64(seed))`` with
``seed = 1809105720 + 1000*cfg + 10*bits + K`` (K = taps for conv1d, else 0).
Activations are drawn first, then each layer's weights in layer order.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Tuple

import numpy as np

SEED_BASE = 1809105720


def seed_for(cfg: int, bits: int, taps: int = 0) -> int:
    return SEED_BASE + 1000 * cfg + 10 * bits + taps


def value_range(bits: int, signed: bool) -> Tuple[int, int]:
    """Inclusive range of a b-bit two's-complement (signed) or unsigned integer."""
    if signed:
        return -(1 << (bits - 1)), (1 << (bits - 1)) - 1
    return 0, (1 << bits) - 1


def uniform(rng: np.random.Generator, shape, bits: int, signed: bool) -> np.ndarray:
    lo, hi = value_range(bits, signed)
    return rng.integers(lo, hi + 1, size=shape, dtype=np.int64).astype(np.int32)


def half_extremes(rng: np.random.Generator, shape, bits: int, signed: bool) -> np.ndarray:
    """Each element independently: with probability 1/2 one of the two range ends
    (each equally likely), otherwise uniform over the whole range."""
    lo, hi = value_range(bits, signed)
    full = rng.integers(lo, hi + 1, size=shape, dtype=np.int64)
    ends = np.where(rng.integers(0, 2, size=shape) == 0, lo, hi)
    pick = rng.integers(0, 2, size=shape) == 0
    return np.where(pick, ends, full).astype(np.int32)


@dataclass(frozen=True)
class Conv2dShape:
    N: int
    C: int
    H: int
    W: int
    M: int
    KH: int
    KW: int
    stride_h: int = 1
    stride_w: int = 1
    pad_h: int = 0
    pad_w: int = 0

    def as_tuple(self) -> Tuple[int, ...]:
        return (self.N, self.C, self.H, self.W, self.M, self.KH, self.KW,
                self.stride_h, self.stride_w, self.pad_h, self.pad_w)


@dataclass
class Conv2dCase:
    cfg: int
    bits: int
    shape: Conv2dShape
    x_signed: bool
    w_signed: bool
    x: np.ndarray          # int32, N x C x H x W, values within b bits
    w: np.ndarray          # int32, M x C x KH x KW
    seed: int = 0


@dataclass
class Conv1dCase:
    bits: int
    taps: int
    x: np.ndarray          # int32, n values, unsigned b-bit
    k: np.ndarray          # int32, K values, unsigned b-bit, natural order
    seed: int = 0


@dataclass
class StackCase:
    bits: int
    layers: List[Conv2dShape]
    x: np.ndarray          # int32, unsigned b-bit input image batch
    ws: List[np.ndarray] = field(default_factory=list)   # int32 signed b-bit weights
    seed: int = 0


SINGLE = Conv2dShape(1, 16, 16, 16, 16, 3, 3, 1, 1, 1, 1)
MID = Conv2dShape(8, 128, 56, 56, 128, 3, 3, 1, 1, 1, 1)
STRESS = Conv2dShape(4, 256, 28, 28, 256, 3, 3, 1, 1, 1, 1)
CONV1D_N = 1 << 20

# AlexNet-shaped stack on 224x224x3, batch 16: five conv layers, no pooling (only
# ReLU + requantisation sits between layers), so every layer after the first is 55x55.
ALEXNET_LAYERS = [
    Conv2dShape(16, 3, 224, 224, 96, 11, 11, 4, 4, 2, 2),
    Conv2dShape(16, 96, 55, 55, 256, 5, 5, 1, 1, 2, 2),
    Conv2dShape(16, 256, 55, 55, 384, 3, 3, 1, 1, 1, 1),
    Conv2dShape(16, 384, 55, 55, 384, 3, 3, 1, 1, 1, 1),
    Conv2dShape(16, 384, 55, 55, 256, 3, 3, 1, 1, 1, 1),
]

# VGG-B (configuration B of Simonyan and Zisserman): ten 3x3 convolutions, stride 1,
# pad 1; a 2x2 max-pool halves the size after layers 2, 4, 6 and 8 (the pools are not
# part of these single-layer workloads).
VGGB_LAYERS = [
    Conv2dShape(1, 3, 224, 224, 64, 3, 3, 1, 1, 1, 1),
    Conv2dShape(1, 64, 224, 224, 64, 3, 3, 1, 1, 1, 1),
    Conv2dShape(1, 64, 112, 112, 128, 3, 3, 1, 1, 1, 1),
    Conv2dShape(1, 128, 112, 112, 128, 3, 3, 1, 1, 1, 1),
    Conv2dShape(1, 128, 56, 56, 256, 3, 3, 1, 1, 1, 1),
    Conv2dShape(1, 256, 56, 56, 256, 3, 3, 1, 1, 1, 1),
    Conv2dShape(1, 256, 28, 28, 512, 3, 3, 1, 1, 1, 1),
    Conv2dShape(1, 512, 28, 28, 512, 3, 3, 1, 1, 1, 1),
    Conv2dShape(1, 512, 14, 14, 512, 3, 3, 1, 1, 1, 1),
    Conv2dShape(1, 512, 14, 14, 512, 3, 3, 1, 1, 1, 1),
]

BITS_SWEEP = {1: [4], 2: list(range(1, 9)), 3: list(range(1, 9)), 4: list(range(2, 9)), 5: [2, 4, 8],
              6: list(range(8, 1, -1))}


def conv2d_case(cfg: int, bits: int, shape: Conv2dShape = None) -> Conv2dCase:
    """Workloads 1, 3 and 4 (``shape`` overrides the size, keeping the value recipe)."""
    seed = seed_for(cfg, bits)
    rng = np.random.Generator(np.random.PCG64(seed))
    if cfg == 1:
        shp, xs, ws, gen = SINGLE, False, True, uniform
    elif cfg == 3:
        shp, xs, ws, gen = MID, False, True, uniform
    elif cfg == 4:
        shp, xs, ws, gen = STRESS, True, True, half_extremes
    else:
        raise ValueError(f"workload {cfg} is not a single conv2d layer")
    if shape is not None:
        shp = shape
    x = gen(rng, (shp.N, shp.C, shp.H, shp.W), bits, xs)
    w = gen(rng, (shp.M, shp.C, shp.KH, shp.KW), bits, ws)
    return Conv2dCase(cfg, bits, shp, xs, ws, x, w, seed)


def conv1d_case(bits: int, taps: int, n: int = CONV1D_N) -> Conv1dCase:
    """Workload 2: unsigned b-bit input of n values and an unsigned b-bit kernel."""
    seed = seed_for(2, bits, taps)
    rng = np.random.Generator(np.random.PCG64(seed))
    x = uniform(rng, (n,), bits, False)
    k = uniform(rng, (taps,), bits, False)
    return Conv1dCase(bits, taps, x, k, seed)


def stack_case(bits: int, batch: int = None, layers: List[Conv2dShape] = None) -> StackCase:
    """Workload 5: unsigned b-bit input image, signed b-bit weights per layer."""
    seed = seed_for(5, bits)
    rng = np.random.Generator(np.random.PCG64(seed))
    lys = list(layers if layers is not None else ALEXNET_LAYERS)
    if batch is not None:
        lys = [Conv2dShape(batch, *l.as_tuple()[1:]) for l in lys]
    first = lys[0]
    x = uniform(rng, (first.N, first.C, first.H, first.W), bits, False)
    ws = [uniform(rng, (l.M, l.C, l.KH, l.KW), bits, True) for l in lys]
    return StackCase(bits, lys, x, ws, seed)


def vggb_case(layer: int, bits: int, batch: int = 1) -> Conv2dCase:
    """Workload 6: VGG-B convolution layer ``layer`` (0-9), signed b-bit activations and
    weights, uniform over the range."""
    seed = seed_for(6, bits, layer)
    rng = np.random.Generator(np.random.PCG64(seed))
    shp = VGGB_LAYERS[layer]
    if batch != shp.N:
        shp = Conv2dShape(batch, *shp.as_tuple()[1:])
    x = uniform(rng, (shp.N, shp.C, shp.H, shp.W), bits, True)
    w = uniform(rng, (shp.M, shp.C, shp.KH, shp.KW), bits, True)
    return Conv2dCase(6, bits, shp, True, True, x, w, seed)
