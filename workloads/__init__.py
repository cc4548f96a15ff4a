"""Seeded synthetic workloads for the split-FFT convolution.

This module only draws random arrays of the right shapes and distributions.
It holds none of the method's arithmetic, so both the CPU oracle tests and
the GPU path tests can use it without sharing any computation.

Recipe (one ``numpy.random.default_rng(seed)`` generator per layer, draws in
the order x, w, b, each drawn in float64 and rounded once to float32):

* layer 1x3x32x32 -> 16, 3x3 kernel: x ~ U[-1, 1], w ~ N(0, sqrt(2/(Cin*K*K))),
  bias zero.
* single VGG-style layers (224^2 x 64, 112^2 x 128, 56^2 x 256 with 5x5):
  x = max(N(0,1), 0) (half zeros, as after a ReLU), w He-normal (fan-in),
  no bias.
* VGG-16-style stack: x ~ U[0, 1] at 3x224x224, 13 3x3 layers with
  He-normal weights and bias ~ U(-1/sqrt(Cin*9), +1/sqrt(Cin*9)).

The paper evaluates on VGG16's convolution layers without naming a dataset;
these synthetic tensors stand in for ImageNet activations and trained
weights, with the same shapes.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import numpy as np


@dataclasses.dataclass(frozen=True)
class Layer:
    """Shape of one stride-1 'same' convolution layer."""

    n: int
    cin: int
    h: int
    w: int
    cout: int
    k: int
    x_dist: str = "relu_normal"   # "uniform_pm1" | "relu_normal" | "uniform_01"
    bias: str = "none"            # "none" | "zero" | "uniform_fanin"
    relu: bool = False

    @property
    def direct_flops(self) -> int:
        """Multiply-adds of the direct convolution, counted as 2 flops each."""
        return 2 * self.n * self.cout * self.h * self.w * self.cin * self.k * self.k


# The five workloads.  "tiles" lists the tile sizes T each one is run with
# (FFT size L = T + K - 1); an empty list means the plan chooses.
CONFIGS = {
    "c1_32x3": dict(layer=Layer(1, 3, 32, 32, 16, 3, "uniform_pm1", "zero"), tiles=[6]),
    "c2_224x64": dict(layer=Layer(1, 64, 224, 224, 64, 3), tiles=[6, 14, 30]),
    "c3_112x128": dict(layer=Layer(8, 128, 112, 112, 128, 3), tiles=[14, 30]),
    "c4_56x256_k5": dict(layer=Layer(16, 256, 56, 56, 256, 5), tiles=[12, 28]),
}

# VGG-16 convolution stack: (cin, cout, spatial) per layer; 2x2 max-pool
# after the layers whose index (1-based) is in VGG_POOL_AFTER.
VGG16_LAYERS = [
    (3, 64, 224), (64, 64, 224),
    (64, 128, 112), (128, 128, 112),
    (128, 256, 56), (256, 256, 56), (256, 256, 56),
    (256, 512, 28), (512, 512, 28), (512, 512, 28),
    (512, 512, 14), (512, 512, 14), (512, 512, 14),
]
VGG_POOL_AFTER = (2, 4, 7, 10, 13)
VGG_BATCH = 32


def _draw_x(rng: np.random.Generator, shape, dist: str) -> np.ndarray:
    if dist == "uniform_pm1":
        a = rng.uniform(-1.0, 1.0, size=shape)
    elif dist == "relu_normal":
        a = np.maximum(rng.standard_normal(size=shape), 0.0)
    elif dist == "uniform_01":
        a = rng.uniform(0.0, 1.0, size=shape)
    else:
        raise ValueError(f"unknown input distribution {dist!r}")
    return a.astype(np.float32)


def _draw_w(rng: np.random.Generator, cout: int, cin: int, k: int) -> np.ndarray:
    std = math.sqrt(2.0 / (cin * k * k))
    return (rng.standard_normal(size=(cout, cin, k, k)) * std).astype(np.float32)


def _draw_b(rng: np.random.Generator, cout: int, cin: int, k: int, kind: str) -> Optional[np.ndarray]:
    if kind == "none":
        return None
    if kind == "zero":
        return np.zeros(cout, dtype=np.float32)
    if kind == "uniform_fanin":
        lim = 1.0 / math.sqrt(cin * k * k)
        return rng.uniform(-lim, lim, size=cout).astype(np.float32)
    raise ValueError(f"unknown bias kind {kind!r}")


def make_layer(layer: Layer, seed: int = 0):
    """Return float32 (x, w, b) for ``layer``; b is None when the layer has no bias."""
    rng = np.random.default_rng(seed)
    x = _draw_x(rng, (layer.n, layer.cin, layer.h, layer.w), layer.x_dist)
    w = _draw_w(rng, layer.cout, layer.cin, layer.k)
    b = _draw_b(rng, layer.cout, layer.cin, layer.k, layer.bias)
    return x, w, b


def make_config(name: str, seed: int = 0):
    return make_layer(CONFIGS[name]["layer"], seed)


def make_random_bias(cout: int, cin: int, k: int, seed: int) -> np.ndarray:
    """A seeded nonzero bias, for runs that exercise the fused bias+ReLU epilogue."""
    rng = np.random.default_rng(seed)
    return _draw_b(rng, cout, cin, k, "uniform_fanin")


def make_vgg16(batch: int = VGG_BATCH, seed: int = 0):
    """Input batch and per-layer (w, b) for the 13-layer VGG-16 stack.

    Returns (x, layers) with layers a list of (w, b) float32 pairs.
    """
    rng = np.random.default_rng(seed)
    x = _draw_x(rng, (batch, 3, 224, 224), "uniform_01")
    layers: List = []
    for cin, cout, _ in VGG16_LAYERS:
        w = _draw_w(rng, cout, cin, 3)
        b = _draw_b(rng, cout, cin, 3, "uniform_fanin")
        layers.append((w, b))
    return x, layers


def small_layer(n, cin, h, w, cout, k, seed=0, dist="uniform_pm1"):
    """A small random layer for edge-case tests (ragged tiles, tiny channels)."""
    rng = np.random.default_rng(seed)
    x = _draw_x(rng, (n, cin, h, w), dist)
    wt = _draw_w(rng, cout, cin, k)
    return x, wt
