"""Seeded synthetic inputs for the N-D Winograd layers.

This module is shared by the oracle tests, the GPU parity tests and the bench.
It holds shapes, value distributions and a seeded generator only: no
convolution, transform or reduction arithmetic of the method lives here.

Recipe (one per layer): a ``torch.Generator('cpu')`` seeded with ``seed`` draws
the input ``x`` first and the weights ``w`` second, both in float32.

* ``normal``       x ~ N(0, 1)
* ``relu_normal``  x = max(0, N(0, 1))   (a post-activation feature map)
* ``uniform``      x ~ U(0, 1)
* ``he``           w ~ N(0, 2 / (C * r**N)), He-normal over the receptive field
* ``int2``         integers uniform in [-2, 2] (exactness checks)

The five layer families mirror the paper's workloads: C3D-style 3x3x3 video
layers (§3.3), the 2-D special case (§3.2), a volumetric 128^3 layer and the
C3D eight-layer stack.  No dataset is used; random tensors of the same shape
and value range stand in for video frames, ImageNet images and trained
weights.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Tuple

import numpy as np

__all__ = [
    "LayerSpec", "StackSpec", "PoolSpec", "CONFIGS", "C3D_STACK",
    "draw_layer", "draw_stack", "draw_tensor", "direct_flops",
]


@dataclass(frozen=True)
class LayerSpec:
    """One N-D convolution layer and the Winograd tile it is run with."""

    name: str
    N: int                     # number of spatial axes
    m: int                     # output-tile extent per axis
    r: int                     # kernel extent per axis
    batch: int
    C: int                     # input channels
    K: int                     # output channels (kernels)
    X: Tuple[int, ...]         # input spatial extents, outer to inner
    pad: int = 0               # symmetric zero padding per axis
    x_dist: str = "normal"
    w_dist: str = "normal"
    relu: bool = False
    points: Tuple = None       # interpolation points; None = library default
    leaky: float = None        # leaky ReLU slope (activation v or slope * v); None = off
    tile: Tuple = None         # per-axis output tiles (eq. 4, one triple per axis); None = m on every axis

    def with_(self, **kw) -> "LayerSpec":
        return replace(self, **kw)

    @property
    def x_shape(self):
        return (self.batch, self.C) + tuple(self.X)

    @property
    def w_shape(self):
        return (self.K, self.C) + (self.r,) * self.N

    @property
    def out_spatial(self):
        return tuple(x + 2 * self.pad - self.r + 1 for x in self.X)


@dataclass(frozen=True)
class PoolSpec:
    window: Tuple[int, int, int]   # max-pool window = stride, floor rounding


@dataclass(frozen=True)
class StackSpec:
    """A stack of 3x3x3 pad-1 layers with ReLU, interleaved with max-pools."""

    name: str
    batch: int
    C_in: int
    X: Tuple[int, int, int]
    widths: Tuple[int, ...]
    pools: dict = field(default_factory=dict)   # layer index -> PoolSpec
    m: int = 2
    x_dist: str = "uniform"

    def layers(self):
        """Yield (LayerSpec, PoolSpec-or-None) in order, shapes propagated."""
        X = tuple(self.X)
        C = self.C_in
        for i, K in enumerate(self.widths):
            spec = LayerSpec(name=f"{self.name}.conv{i + 1}", N=3, m=self.m, r=3,
                             batch=self.batch, C=C, K=K, X=X, pad=1,
                             x_dist=self.x_dist, w_dist="he", relu=True)
            pool = self.pools.get(i)
            yield spec, pool
            X = spec.out_spatial
            if pool is not None:
                X = tuple(x // p for x, p in zip(X, pool.window))
            C = K


# The five workloads the throughput metric is quoted on.
CONFIGS = {
    1: LayerSpec("f2x3_3d_c16", N=3, m=2, r=3, batch=1, C=16, K=16, X=(16, 16, 16),
                 pad=0, x_dist="normal", w_dist="normal"),
    2: LayerSpec("f2x3_3d_c64k128", N=3, m=2, r=3, batch=8, C=64, K=128, X=(16, 56, 56),
                 pad=1, x_dist="relu_normal", w_dist="he"),
    3: LayerSpec("f4x3_2d_c256", N=2, m=4, r=3, batch=64, C=256, K=256, X=(56, 56),
                 pad=1, x_dist="relu_normal", w_dist="he"),
    4: LayerSpec("f4x3_3d_vol128", N=3, m=4, r=3, batch=1, C=32, K=32, X=(128, 128, 128),
                 pad=1, x_dist="uniform", w_dist="he"),
}

C3D_STACK = StackSpec(
    name="c3d", batch=4, C_in=3, X=(16, 112, 112),
    widths=(64, 128, 256, 256, 512, 512, 512, 512),
    pools={0: PoolSpec((1, 2, 2)), 1: PoolSpec((2, 2, 2)), 3: PoolSpec((2, 2, 2)),
           5: PoolSpec((2, 2, 2)), 7: PoolSpec((2, 2, 2))},
    m=2, x_dist="uniform")


def fig4_layers(batch=200, X=224, depth=3):
    """Stand-in for the paper's 2-D benchmark (§4.4, Fig. 4): a 224 x 224 image
    through three unpadded 4 x 4 layers of 32 channels and 32 kernels (no
    activation is stated; none is applied), here with F(5^2, 4^2).  Layer i + 1
    takes layer i's output; random inputs stand in for the ImageNet images."""
    out = []
    for i in range(depth):
        out.append(LayerSpec(f"fig4_l{i + 1}_b{batch}", N=2, m=5, r=4, batch=batch, C=32, K=32,
                             X=(X, X), pad=0, x_dist="uniform", w_dist="he"))
        X -= 3
    return out


def _gen(seed):
    import torch
    return torch.Generator("cpu").manual_seed(int(seed))


def draw_tensor(gen, shape, dist, fan_in=1):
    """Draw one float32 tensor of ``shape`` from ``dist`` with generator ``gen``."""
    import torch
    shape = tuple(int(s) for s in shape)
    if dist == "normal":
        t = torch.randn(shape, generator=gen, dtype=torch.float32)
    elif dist == "relu_normal":
        t = torch.randn(shape, generator=gen, dtype=torch.float32).clamp_(min=0.0)
    elif dist == "uniform":
        t = torch.rand(shape, generator=gen, dtype=torch.float32)
    elif dist == "he":
        t = torch.randn(shape, generator=gen, dtype=torch.float32)
        t.mul_(float(np.sqrt(2.0 / fan_in)))
    elif dist == "int2":
        t = torch.randint(-2, 3, shape, generator=gen).to(torch.float32)
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    return t.numpy()


def draw_layer(spec: LayerSpec, seed: int):
    """Return (x, w) as float32 numpy arrays for one layer; x drawn first."""
    g = _gen(seed)
    x = draw_tensor(g, spec.x_shape, spec.x_dist)
    w = draw_tensor(g, spec.w_shape, spec.w_dist, fan_in=spec.C * spec.r ** spec.N)
    return x, w


def draw_stack(stack: StackSpec, seed: int):
    """Return (x, [w1..wL]) for a stack; x first, then each layer's weights."""
    g = _gen(seed)
    x = draw_tensor(g, (stack.batch, stack.C_in) + tuple(stack.X), stack.x_dist)
    ws = []
    for spec, _ in stack.layers():
        ws.append(draw_tensor(g, spec.w_shape, spec.w_dist, fan_in=spec.C * spec.r ** spec.N))
    return x, ws


def direct_flops(spec: LayerSpec) -> int:
    """Direct-convolution FLOP count 2*n*K*C*r^N*prod(Y), padded zeros counted."""
    n = 2 * spec.batch * spec.K * spec.C * spec.r ** spec.N
    for y in spec.out_spatial:
        n *= y
    return int(n)
