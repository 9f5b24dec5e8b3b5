"""GPU parity of the weight gradient (wino_weight_gradient) against the fp64
oracle on the same seeded inputs, on every output.

Bar: normalised max error |dw - dw_ref| / sum |dy| |x~| <= 1e-4.  Unlike the
forward (a sum over C channels), every dw entry sums over all tiles of the
batch: an fp32 MFMA accumulator chain adds up to 64 * (tile blocks per split)
products (3,136 for the F(2^3) C = 64, K = 128 layer at batch 8), whose
first-order rounding bound is about that count times 2^-24 (1.9e-4) of the
summed magnitudes, and a random-sign walk about its square root times 2^-24
(3.4e-6); the bar sits between them.
"""
import math

import numpy as np
import pytest

from gpu_util import log, require_gpu
from oracle.metric import normalised_error
from oracle.wgrad import direct_wgrad
from workloads import CONFIGS

pytestmark = pytest.mark.gpu

TOL_WGRAD = 1e-4

# (name, N, m, r, batch, C, K, X, pad)
WG = [
    ("f2x3_3d", 3, 2, 3, 2, 24, 40, (6, 13, 15), 1),
    ("f2x3_3d_c70k90", 3, 2, 3, 1, 70, 90, (9, 10, 12), 1),
    ("f2x3_2d_pad0", 2, 2, 3, 2, 10, 33, (19, 14), 0),
    ("f2x3_2d_pad2", 2, 2, 3, 3, 5, 7, (11, 9), 2),
    ("f2x3_3d_one_tile", 3, 2, 3, 1, 3, 2, (3, 3, 3), 0),
    ("f4x3_2d", 2, 4, 3, 3, 36, 70, (17, 23), 1),
    ("f4x3_2d_c130", 2, 4, 3, 2, 130, 20, (12, 9), 1),
    # edges: one channel and one kernel, a pad wider than r - 1 (windows
    # entirely in the padding), odd extents (partial tiles on every axis)
    ("f2x3_3d_c1k1", 3, 2, 3, 1, 1, 1, (5, 4, 6), 1),
    ("f2x3_2d_pad3", 2, 2, 3, 2, 3, 5, (6, 7), 3),
    ("f2x3_3d_odd", 3, 2, 3, 3, 5, 66, (7, 5, 9), 0),
    ("f4x3_2d_c1", 2, 4, 3, 1, 1, 9, (10, 13), 2),
    # V in 16-tile blocks: F(4^3) and the alpha = 8 sizes of Table 1, F(3,2)
    ("f4x3_3d", 3, 4, 3, 1, 20, 24, (13, 11, 17), 1),
    ("f4x3_3d_c40k70", 3, 4, 3, 2, 40, 70, (9, 8, 12), 2),
    # F(4^3) with whole tiles on the last axis (16-byte row loads of dy) and
    # partial tiles on the other two
    ("f4x3_3d_rows", 3, 4, 3, 2, 6, 10, (7, 9, 16), 1),
    ("f5x4_2d", 2, 5, 4, 2, 9, 20, (23, 31), 1),
    ("f4x5_2d", 2, 4, 5, 2, 12, 19, (21, 26), 2),
    ("f3x6_2d", 2, 3, 6, 1, 20, 33, (25, 19), 0),
    ("f3x2_2d", 2, 3, 2, 3, 17, 40, (20, 23), 0),
    ("f3x2_3d", 3, 3, 2, 2, 10, 20, (7, 9, 8), 1),
]


def run_wgrad(N, m, r, batch, C, K, X, pad, x_fn, dy_fn, name, points=None):
    torch = require_gpu()
    from paper_1611_06565_amd.wino import Plan
    log(f"[gpu] wgrad {name} N={N} m={m} r={r} C={C} K={K} X={X} batch={batch} pad={pad} points={points}")
    plan = Plan(N, m, r, C, K, [batch] + list(X), pad=pad, points=points)
    assert plan.weight_gradient_workspace_bytes > 0
    x = x_fn(plan.input_shape)
    dy = dy_fn(plan.output_shape)
    dw = plan.weight_gradient(torch.from_numpy(x).cuda(), torch.from_numpy(dy).cuda())
    torch.cuda.synchronize()
    return dw.cpu().numpy(), x, dy


def _check(dw, x, dy, r, pad):
    ref, den = direct_wgrad(x, dy, r, pad)
    err = normalised_error(dw, ref, den)
    log(f"  max err {err['max']:.3e} p99.99 {err['p9999']:.3e} at {err['argmax']}")
    assert err["nonfinite"] == 0
    assert err["max"] <= TOL_WGRAD, err


@pytest.mark.parametrize("case", WG, ids=lambda c: c[0])
def test_wgrad_full_output(case):
    name, N, m, r, batch, C, K, X, pad = case
    rng = np.random.default_rng(41)
    dw, x, dy = run_wgrad(N, m, r, batch, C, K, X, pad,
                          lambda s: rng.standard_normal(s).astype(np.float32),
                          lambda s: rng.standard_normal(s).astype(np.float32), name)
    _check(dw, x, dy, r, pad)


@pytest.mark.parametrize("N,m,points", [(3, 2, (0, 0.5, -0.5)), (2, 4, (0, 1, -1, 1.0 / 3.0, -1.0 / 3.0)),
                                         (2, 4, (0, 2, -2, 0.5, -0.5))],
                         ids=["f23_half_pts", "f43_paper_pts", "f43_searched_pts"])
def test_wgrad_caller_points(N, m, points):
    # F(r, m) is built on the caller's points as well (its B^T is again the
    # forward's, checked exactly by the plan)
    rng = np.random.default_rng(43)
    X = (6, 9, 11) if N == 3 else (17, 14)
    dw, x, dy = run_wgrad(N, m, 3, 2, 12, 20, X, 1,
                          lambda s: rng.standard_normal(s).astype(np.float32),
                          lambda s: rng.standard_normal(s).astype(np.float32), "points", points)
    _check(dw, x, dy, 3, 1)


def test_wgrad_integer_inputs_bitwise_exact():
    # F(2^3): F(3, 2)'s matrices hold 0, +-1 and +-1/2 only, so small-integer
    # data keeps every intermediate an exact fp32 value
    rng = np.random.default_rng(6)
    dw, x, dy = run_wgrad(3, 2, 3, 2, 12, 20, (5, 9, 7), 1,
                          lambda s: rng.integers(-2, 3, size=s).astype(np.float32),
                          lambda s: rng.integers(-2, 3, size=s).astype(np.float32), "int")
    ref, _ = direct_wgrad(x, dy, 3, 1, with_den=False)
    assert np.array_equal(dw, ref.astype(np.float32))


def test_wgrad_determinism_bitwise():
    rng = np.random.default_rng(7)
    shp = {}
    x_fn = lambda s: shp.setdefault("x", rng.standard_normal(s).astype(np.float32))   # noqa: E731
    dy_fn = lambda s: shp.setdefault("dy", rng.standard_normal(s).astype(np.float32))  # noqa: E731
    a, _, _ = run_wgrad(3, 2, 3, 2, 24, 40, (6, 13, 15), 1, x_fn, dy_fn, "det1")
    b, _, _ = run_wgrad(3, 2, 3, 2, 24, 40, (6, 13, 15), 1, x_fn, dy_fn, "det2")
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_wgrad_full_size():
    # the F(2^3) C = 64, K = 128, 16 x 56 x 56 layer at batch 8, every output
    spec = CONFIGS[2]
    rng = np.random.default_rng(9)
    dw, x, dy = run_wgrad(spec.N, spec.m, spec.r, spec.batch, spec.C, spec.K, spec.X, spec.pad,
                          lambda s: np.maximum(rng.standard_normal(s, dtype=np.float32), 0),
                          lambda s: rng.standard_normal(s, dtype=np.float32) * math.sqrt(1.0 / spec.K),
                          spec.name)
    _check(dw, x, dy, spec.r, spec.pad)


def test_wgrad_f4x3_3d_full_size():
    # the F(4^3) C = K = 32, 128^3 layer (V in 16-tile blocks), every output
    spec = CONFIGS[4]
    rng = np.random.default_rng(10)
    dw, x, dy = run_wgrad(spec.N, spec.m, spec.r, spec.batch, spec.C, spec.K, spec.X, spec.pad,
                          lambda s: rng.random(s, dtype=np.float32),
                          lambda s: rng.standard_normal(s, dtype=np.float32) * math.sqrt(1.0 / spec.K),
                          spec.name)
    _check(dw, x, dy, spec.r, spec.pad)
