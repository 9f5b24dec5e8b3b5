"""Invariants of the HIP forward that need no oracle value: each follows from
the definition of the layer (eq. 2) and from the tile decomposition of §3.

* Translation: with no padding, dropping the first m input planes of an axis
  shifts the output by m planes along it.  The tiles of the shifted input are
  the old tiles one step on, so every output is formed by the same arithmetic
  on the same values and the outputs must agree bit for bit.
* Batch independence: a sample's output does not depend on the other samples
  of the batch, bit for bit.
* Scaling: y(2x) = 2 y(x) bit for bit (doubling is exact in fp32 and commutes
  with every sum and product of the path); linearity y(a x1 + b x2) = a y(x1)
  + b y(x2) within the layer's bar.
* One-hot input: a single unit input value at p in channel c gives, at output
  o, the kernel tap w[k][c][p + pad - o] (eq. 2 correlates without a flip), so
  the output holds the kernel mirrored about p; a flipped kernel fails.

Products are run unsplit (WINO_NO_SPLIT) where bitwise equality is asserted:
a split block sums its partial products in another order than a whole one,
and which blocks are split depends on the grid.
"""
import numpy as np
import pytest

from gpu_util import log, require_gpu, run_layer, tol
from oracle.direct import direct_blas
from workloads import LayerSpec, draw_layer

pytestmark = pytest.mark.gpu

# one layer per product kernel: k_gemm_acc (F(2^3), F(2^2)), k_gemm_acc4
# (F(4^2)), k_fused43 and k_input_split + k_gemm_inv (F(4^3)), the per-axis
# F(2,3) x F(4,3)^2 kernels and k_gemm_inv on an alpha = 8 2-D size
PATHS = [
    (LayerSpec("inv_f2x3_3d", N=3, m=2, r=3, batch=2, C=20, K=70, X=(9, 12, 14), pad=0,
               x_dist="normal", w_dist="he"), {}),
    (LayerSpec("inv_f2x3_2d", N=2, m=2, r=3, batch=3, C=12, K=40, X=(23, 19), pad=0,
               x_dist="normal", w_dist="he"), {}),
    (LayerSpec("inv_f4x2", N=2, m=4, r=3, batch=2, C=36, K=45, X=(26, 30), pad=0,
               x_dist="normal", w_dist="he"), {}),
    (LayerSpec("inv_f4x3_fused", N=3, m=4, r=3, batch=2, C=20, K=24, X=(14, 13, 17), pad=0,
               x_dist="normal", w_dist="he"), {"fuse": True}),
    (LayerSpec("inv_f4x3_two_stage", N=3, m=4, r=3, batch=2, C=20, K=24, X=(14, 13, 17), pad=0,
               x_dist="normal", w_dist="he"), {"fuse": False}),
    (LayerSpec("inv_aniso_244", N=3, m=2, r=3, batch=2, C=12, K=20, X=(10, 15, 13), pad=0,
               x_dist="normal", w_dist="he", tile=(2, 4, 4)), {}),
    (LayerSpec("inv_f5x4_2d", N=2, m=5, r=4, batch=2, C=8, K=12, X=(27, 24), pad=0,
               x_dist="normal", w_dist="he"), {}),
    # Table 1's sizes in 3-D: k_gemm_inv with 8 waves (F(3^3, 2^3)) and k_gemm_a8
    (LayerSpec("inv_f3x2_3d", N=3, m=3, r=2, batch=2, C=10, K=20, X=(10, 9, 11), pad=0,
               x_dist="normal", w_dist="he"), {}),
    (LayerSpec("inv_f5x4_3d", N=3, m=5, r=4, batch=2, C=6, K=20, X=(14, 12, 13), pad=0,
               x_dist="normal", w_dist="he"), {}),
]
IDS = [p[0].name for p in PATHS]


def _run(spec, x, w, kw):
    y, plan = run_layer(spec, x, w, split=False, **kw)
    if "fuse" in kw:
        assert plan.desc["fused"] == (1 if kw["fuse"] else 0)
    return y


def _bits(a):
    return np.ascontiguousarray(a).view(np.uint32)


def _tile_of(spec, axis):
    return spec.tile[axis] if spec.tile else spec.m


@pytest.mark.parametrize("spec,kw", PATHS, ids=IDS)
def test_translation_by_tile_is_bitwise(spec, kw):
    x, w = draw_layer(spec, seed=41)
    y = _run(spec, x, w, kw)
    # shift along the first spatial axis (and the last, where the row layout
    # of the input stays the same kind: fewer than 16 tiles per row)
    axes = [0] + ([spec.N - 1] if -(-spec.out_spatial[-1] // _tile_of(spec, spec.N - 1)) < 16 else [])
    for a in axes:
        s = _tile_of(spec, a)
        X2 = tuple(v - s if i == a else v for i, v in enumerate(spec.X))
        sl = [slice(None), slice(None)] + [slice(s, None) if i == a else slice(None) for i in range(spec.N)]
        x2 = np.ascontiguousarray(x[tuple(sl)])
        y2 = _run(spec.with_(X=X2, name=spec.name + f"_shift{a}"), x2, w, kw)
        ref = y[tuple(sl)]
        log(f"  axis {a}: shift {s}, {y2.size} outputs")
        assert y2.shape == ref.shape
        assert np.array_equal(_bits(y2), _bits(ref)), f"axis {a}: shifted output differs"


@pytest.mark.parametrize("spec,kw", PATHS, ids=IDS)
def test_batch_independence_bitwise(spec, kw):
    x, w = draw_layer(spec, seed=42)
    y = _run(spec, x, w, kw)
    for b in range(spec.batch):
        yb = _run(spec.with_(batch=1, name=spec.name + f"_b{b}"), np.ascontiguousarray(x[b:b + 1]), w, kw)
        assert np.array_equal(_bits(yb[0]), _bits(y[b])), f"sample {b} depends on the batch"


@pytest.mark.parametrize("spec,kw", PATHS, ids=IDS)
def test_scaling_bitwise_and_linearity(spec, kw):
    x1, w = draw_layer(spec, seed=43)
    x2, _ = draw_layer(spec, seed=44)
    y1 = _run(spec, x1, w, kw)
    y1d = _run(spec, 2.0 * x1, w, kw)
    assert np.array_equal(_bits(y1d), _bits(2.0 * y1)), "y(2x) != 2 y(x)"
    a, b = np.float32(0.75), np.float32(-1.5)
    xl = (a * x1 + b * x2).astype(np.float32)
    y2 = _run(spec, x2, w, kw)
    yl = _run(spec, xl, w, kw)
    # each side is within the bar of the exact result; the exact results are
    # linear in x, so the difference is within the sum of the three bars
    _, den1 = direct_blas(x1, w, spec.pad)
    _, den2 = direct_blas(x2, w, spec.pad)
    _, denl = direct_blas(xl, w, spec.pad)
    bound = tol(spec) * (denl + abs(float(a)) * den1 + abs(float(b)) * den2)
    diff = np.abs(yl.astype(np.float64) - (float(a) * y1.astype(np.float64) + float(b) * y2.astype(np.float64)))
    log(f"  linearity: max diff / bound {float(np.max(diff / np.maximum(bound, 1e-30))):.3e}")
    assert np.all(diff <= bound)


@pytest.mark.parametrize("spec,kw", PATHS, ids=IDS)
def test_one_hot_gives_the_mirrored_kernel(spec, kw):
    spec = spec.with_(batch=1, pad=1 if spec.r == 3 else 0)
    require_gpu()
    x = np.zeros(spec.x_shape, dtype=np.float32)
    rng = np.random.default_rng(5)
    _, w = draw_layer(spec, seed=45)
    c = int(rng.integers(0, spec.C))
    p = tuple(int(v) // 2 for v in spec.X)
    x[(0, c) + p] = 1.0
    y = _run(spec, x, w, kw)
    Y = spec.out_spatial
    exp = np.zeros((spec.K,) + Y)
    flipped = np.zeros((spec.K,) + Y)     # what a convolution (flipped kernel) would give
    for q in np.ndindex(*(spec.r,) * spec.N):
        o = tuple(pi + spec.pad - qi for pi, qi in zip(p, q))
        if all(0 <= oi < yi for oi, yi in zip(o, Y)):
            exp[(slice(None),) + o] = w[(slice(None), c) + q]
            flipped[(slice(None),) + o] = w[(slice(None), c) + tuple(spec.r - 1 - qi for qi in q)]
    # errors against the largest tap of the channel: outputs away from the
    # window must be near zero, and a flipped or shifted kernel leaves
    # errors of the order of the taps themselves
    scale = float(np.max(np.abs(w[:, c])))
    err = float(np.max(np.abs(y[0] - exp))) / scale
    log(f"  one-hot channel {c} at {p}: max err / max|w| {err:.3e}")
    assert err <= 10 * tol(spec)
    assert float(np.max(np.abs(y[0] - flipped))) / scale > 0.1
