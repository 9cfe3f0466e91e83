"""Seeded synthetic inputs and the layer shapes of the benchmark workloads.

This module holds no arithmetic of the band-limited method: it only draws
activations, filters and output gradients with the shapes and value
statistics of the paper's workloads (CIFAR-sized ResNet-18 / DenseNet-121
3x3 layers, the 3-layer FCN for UCR time series of Sec. 4 and the
supplementary experimental setup), so that the GPU path and the fp64 oracle
are fed the very same fp32 tensors.

Recipe (fixed, so every run regenerates bit-identical inputs):
  * RNG: ``numpy.random.Generator(PCG64(seed))`` with
    ``seed = 1000*config + 10*layer + {0: x, 1: w, 2: dy}``.
  * Values are drawn in fp64 and rounded to fp32 once.
  * Filters: Kaiming-normal, N(0, 2/fan_in) with fan_in = C_in * K**ndim.
  * Output gradients: N(0, 1) of shape [N, C_out, Ho(, Wo)].
  * 2-D activations: N(0, 1) planes smoothed by a separable Gaussian blur
    (taps exp(-k^2 / (2 sigma^2)) for |k| <= ceil(4 sigma), normalised to sum
    one, numpy 'reflect' boundary), optionally followed by ReLU.
  * 1-D activations: a random walk (cumulative sum of N(0, 1) steps) plus
    N(0, 0.1^2) noise, z-normalised per (sample, channel) series.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Layer:
    """One convolution layer: shapes, padding and the activation recipe.

    ``pad`` is (top, bottom, left, right) for 2-D and (lo, hi) for 1-D.
    For 1-D layers ``H`` is the sequence length and ``W`` is 1.
    """

    name: str
    ndim: int
    N: int
    C_in: int
    C_out: int
    H: int
    W: int
    K: int
    pad: tuple
    act: str  # "blur", "blur_relu" or "walk"
    sigma: float = 0.0

    @property
    def out_hw(self):
        if self.ndim == 1:
            return (self.H + self.pad[0] + self.pad[1] - self.K + 1,)
        Hp = self.H + self.pad[0] + self.pad[1]
        Wp = self.W + self.pad[2] + self.pad[3]
        return (Hp - self.K + 1, Wp - self.K + 1)

    def x_shape(self):
        if self.ndim == 1:
            return (self.N, self.C_in, self.H)
        return (self.N, self.C_in, self.H, self.W)

    def w_shape(self):
        return (self.C_out, self.C_in) + (self.K,) * self.ndim

    def dy_shape(self):
        return (self.N, self.C_out) + self.out_hw

    def direct_flops(self):
        """Multiply-add count of the equivalent direct convolution, x2 (one pass)."""
        return 2 * self.N * self.C_in * self.C_out * int(np.prod(self.out_hw)) * self.K ** self.ndim


@dataclass(frozen=True)
class Config:
    index: int
    name: str
    layers: tuple
    rates: tuple = field(default=(0.0, 0.25, 0.5, 0.75))


def _same(K):
    lo = (K - 1) // 2
    return lo, K - 1 - lo


WORKLOADS = {
    1: Config(1, "tiny 2-D layer 3->16 @32x32, batch 2",
              (Layer("tiny_3to16_32", 2, 2, 3, 16, 32, 32, 3, (1, 1, 1, 1), "blur", 1.5),),
              (0.0, 0.5)),
    2: Config(2, "1-D FCN time-series stack, batch 64, length 512",
              (Layer("fcn1_1to128_k8", 1, 64, 1, 128, 512, 1, 8, _same(8), "walk"),
               Layer("fcn2_128to256_k5", 1, 64, 128, 256, 512, 1, 5, _same(5), "walk"),
               Layer("fcn3_256to128_k3", 1, 64, 256, 128, 512, 1, 3, _same(3), "walk"))),
    3: Config(3, "ResNet-18-shaped 3x3 layers at CIFAR resolution, batch 128",
              (Layer("resnet_64_32", 2, 128, 64, 64, 32, 32, 3, (1, 1, 1, 1), "blur_relu", 1.0),
               Layer("resnet_128_16", 2, 128, 128, 128, 16, 16, 3, (1, 1, 1, 1), "blur_relu", 1.0),
               Layer("resnet_256_8", 2, 128, 256, 256, 8, 8, 3, (1, 1, 1, 1), "blur_relu", 1.0),
               Layer("resnet_512_4", 2, 128, 512, 512, 4, 4, 3, (1, 1, 1, 1), "blur_relu", 1.0))),
    4: Config(4, "DenseNet-121-shaped bottleneck 3x3 layers, batch 64, growth 32",
              (Layer("densenet_128to32_32", 2, 64, 128, 32, 32, 32, 3, (1, 1, 1, 1), "blur_relu", 1.0),
               Layer("densenet_128to32_16", 2, 64, 128, 32, 16, 16, 3, (1, 1, 1, 1), "blur_relu", 1.0),
               Layer("densenet_128to32_8", 2, 64, 128, 32, 8, 8, 3, (1, 1, 1, 1), "blur_relu", 1.0))),
    5: Config(5, "large-image layer 64->64 @56x56, batch 32",
              (Layer("large_64_56", 2, 32, 64, 64, 56, 56, 3, (1, 1, 1, 1), "blur", 2.0),),
              (0.0, 0.5, 0.75)),
}


def seed_for(config: int, layer: int, which: str) -> int:
    return 1000 * config + 10 * layer + {"x": 0, "w": 1, "dy": 2}[which]


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def gaussian_taps(sigma: float) -> np.ndarray:
    r = int(math.ceil(4.0 * sigma))
    k = np.arange(-r, r + 1, dtype=np.float64)
    g = np.exp(-(k * k) / (2.0 * sigma * sigma))
    return g / g.sum()


def blur_planes(a: np.ndarray, sigma: float) -> np.ndarray:
    """Separable Gaussian blur over the last two axes (H then W), reflect boundary."""
    g = gaussian_taps(sigma)
    r = (len(g) - 1) // 2
    out = a
    for axis in (-2, -1):
        widths = [(0, 0)] * out.ndim
        widths[axis] = (r, r)
        p = np.pad(out, widths, mode="reflect")
        n = out.shape[axis]
        acc = np.zeros_like(out)
        for t in range(len(g)):
            sl = [slice(None)] * out.ndim
            sl[axis] = slice(t, t + n)
            acc += g[t] * p[tuple(sl)]
        out = acc
    return out


def random_walk_series(rng, n, c, length) -> np.ndarray:
    steps = rng.standard_normal((n, c, length))
    walk = np.cumsum(steps, axis=-1) + 0.1 * rng.standard_normal((n, c, length))
    mu = walk.mean(axis=-1, keepdims=True)
    sd = walk.std(axis=-1, keepdims=True)
    return (walk - mu) / np.where(sd > 0, sd, 1.0)


def make_x(layer: Layer, seed: int) -> np.ndarray:
    rng = _rng(seed)
    if layer.act == "walk":
        a = random_walk_series(rng, layer.N, layer.C_in, layer.H)
    else:
        a = blur_planes(rng.standard_normal(layer.x_shape()), layer.sigma)
        if layer.act == "blur_relu":
            a = np.maximum(a, 0.0)
    return a.astype(np.float32)


def make_w(layer: Layer, seed: int) -> np.ndarray:
    rng = _rng(seed)
    fan_in = layer.C_in * layer.K ** layer.ndim
    return (rng.standard_normal(layer.w_shape()) * math.sqrt(2.0 / fan_in)).astype(np.float32)


def make_dy(layer: Layer, seed: int) -> np.ndarray:
    rng = _rng(seed)
    return rng.standard_normal(layer.dy_shape()).astype(np.float32)


def layer_inputs(config: int, layer_index: int, layer: Layer | None = None):
    """(x, w, dy) fp32 arrays for one layer of a workload, from the fixed seeds."""
    if layer is None:
        layer = WORKLOADS[config].layers[layer_index]
    return (make_x(layer, seed_for(config, layer_index, "x")),
            make_w(layer, seed_for(config, layer_index, "w")),
            make_dy(layer, seed_for(config, layer_index, "dy")))


def random_layer(rng, ndim, max_hw=12, max_c=4, max_n=2, max_k=5):
    """A small random layer (for parity sweeps over odd shapes and paddings)."""
    K = int(rng.integers(1, max_k + 1))
    if ndim == 1:
        L = int(rng.integers(max(K, 1), 4 * max_hw + 1))
        lo, hi = int(rng.integers(0, K)), int(rng.integers(0, K))
        if L + lo + hi < K:
            hi = K - L - lo
        return Layer("rand1d", 1, int(rng.integers(1, max_n + 1)), int(rng.integers(1, max_c + 1)),
                     int(rng.integers(1, max_c + 1)), L, 1, K, (lo, hi), "blur")
    H = int(rng.integers(1, max_hw + 1))
    W = int(rng.integers(1, max_hw + 1))
    pad = tuple(int(rng.integers(0, K)) for _ in range(4))
    pt, pb, pl, pr = pad
    if H + pt + pb < K:
        pb = K - H - pt
    if W + pl + pr < K:
        pr = K - W - pl
    return Layer("rand2d", 2, int(rng.integers(1, max_n + 1)), int(rng.integers(1, max_c + 1)),
                 int(rng.integers(1, max_c + 1)), H, W, K, (pt, pb, pl, pr), "blur")


def random_inputs(layer: Layer, seed: int):
    """Plain N(0,1) fp32 inputs for a random layer."""
    rng = _rng(seed)
    x = rng.standard_normal(layer.x_shape()).astype(np.float32)
    w = rng.standard_normal(layer.w_shape()).astype(np.float32)
    dy = rng.standard_normal(layer.dy_shape()).astype(np.float32)
    return x, w, dy
