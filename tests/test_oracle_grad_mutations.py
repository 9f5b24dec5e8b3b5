"""Planted mistakes in the gradient oracles (CPU only) must be caught by their
pins: each variant below is the oracle's algorithm with one plausible slip (a
missing flip, a transposed kernel, an off-by-one shift or crop, swapped roles
of input and output gradient), and the pin that the real oracle passes
rejects it."""
import itertools

import numpy as np
import pytest

from oracle.adjoint import direct_adjoint
from oracle.direct import direct_blas
from oracle.wgrad import direct_wgrad


def _adjoint_variant(dy, w, pad, slip):
    n, K = dy.shape[:2]
    C, r = w.shape[1], w.shape[2]
    N = dy.ndim - 2
    Y = dy.shape[2:]
    X = tuple(y - 2 * pad + r - 1 for y in Y)
    if slip == "flip":
        w = w[(slice(None), slice(None)) + (slice(None, None, -1),) * N]
    if slip == "transpose":
        w = np.swapaxes(w, 0, 1)
    buf = np.zeros((n, C) + tuple(x + 2 * pad + 1 for x in X))
    for p in itertools.product(range(r), repeat=N):
        sl = (slice(None), slice(None)) + tuple(slice(pi, pi + yi) for pi, yi in zip(p, Y))
        buf[sl] += np.moveaxis(np.tensordot(dy, w[(slice(None), slice(None)) + p], axes=([1], [0])), -1, 1)
    lo = pad + (1 if slip == "crop_shift" else 0)
    return buf[(slice(None), slice(None)) + tuple(slice(lo, lo + x) for x in X)]


def _wgrad_variant(x, dy, r, pad, slip):
    N = x.ndim - 2
    K, C = dy.shape[1], x.shape[1]
    Y = dy.shape[2:]
    xp = np.pad(x, [(0, 0), (0, 0)] + [(pad, pad + 1)] * N)
    dw = np.zeros((K, C) + (r,) * N)
    axes = ([0] + list(range(2, 2 + N)),) * 2
    for p in itertools.product(range(r), repeat=N):
        q = tuple(pi + (1 if slip == "shift" else 0) for pi in p)
        win = xp[(slice(None), slice(None)) + tuple(slice(qi, qi + yi) for qi, yi in zip(q, Y))]
        t = np.tensordot(dy, win, axes=axes)
        if slip == "swap":
            t = np.tensordot(win, dy, axes=axes)
        dw[(slice(None), slice(None)) + p] = t
    if slip == "flip":
        dw = dw[(slice(None), slice(None)) + (slice(None, None, -1),) * N]
    return dw


def _case(seed=0):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((2, 4, 6, 7, 5))
    w = rng.standard_normal((4, 4, 3, 3, 3))     # C = K, so a transposed kernel keeps its shape
    y, _ = direct_blas(x, w, 1, with_den=False)
    dy = rng.standard_normal(y.shape)
    return x, w, y, dy


def _identity_holds(lhs, rhs, scale):
    return abs(lhs - rhs) <= 1e-9 * scale


def test_real_gradient_oracles_pass_the_identity():
    x, w, y, dy = _case()
    dx, _ = direct_adjoint(dy, w, 1)
    dw, _ = direct_wgrad(x, dy, 3, 1)
    scale = float(np.sum(np.abs(y * dy)))
    assert _identity_holds(np.sum(y * dy), np.sum(x * dx), scale)
    assert _identity_holds(np.sum(y * dy), np.sum(w * dw), scale)


@pytest.mark.parametrize("slip", ["flip", "transpose", "crop_shift"])
def test_adjoint_mutations_caught(slip):
    x, w, y, dy = _case(1)
    dx = _adjoint_variant(dy, w, 1, slip)
    assert dx.shape == x.shape
    assert not _identity_holds(np.sum(y * dy), np.sum(x * dx), float(np.sum(np.abs(y * dy))))


def test_adjoint_variant_without_slip_matches():
    x, w, y, dy = _case(2)
    assert np.allclose(_adjoint_variant(dy, w, 1, None), direct_adjoint(dy, w, 1)[0], rtol=0, atol=1e-12)


@pytest.mark.parametrize("slip", ["shift", "swap", "flip"])
def test_wgrad_mutations_caught(slip):
    x, w, y, dy = _case(3)
    dw = _wgrad_variant(x, dy, 3, 1, slip)
    assert dw.shape == w.shape
    assert not _identity_holds(np.sum(y * dy), np.sum(w * dw), float(np.sum(np.abs(y * dy))))


def test_wgrad_variant_without_slip_matches():
    x, w, y, dy = _case(4)
    assert np.allclose(_wgrad_variant(x, dy, 3, 1, None), direct_wgrad(x, dy, 3, 1)[0], rtol=0, atol=1e-12)
