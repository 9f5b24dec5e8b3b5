"""Pins of the data-gradient oracle (oracle/adjoint.py) against facts outside it."""
import itertools

import numpy as np
import pytest
import torch

from oracle.adjoint import direct_adjoint, direct_adjoint_sampled, in_extent
from oracle.direct import direct_blas, direct_naive, out_extent


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


@pytest.mark.parametrize("N,r,pad", [(1, 3, 0), (2, 3, 1), (2, 3, 0), (3, 3, 1), (3, 3, 2),
                                     (2, 4, 1), (2, 2, 0), (2, 5, 2), (2, 6, 4), (2, 3, 3)])
def test_inner_product_identity(N, r, pad):
    # the defining property of an adjoint: <A x, dy> = <x, A^T dy>
    X = (9, 7, 6)[:N]
    C, K, n = 3, 4, 2
    x = _rand((n, C) + X, 1)
    w = _rand((K, C) + (r,) * N, 2)
    y, _ = direct_blas(x, w, pad, with_den=False)
    dy = _rand(y.shape, 3)
    dx, _ = direct_adjoint(dy, w, pad)
    assert dx.shape == x.shape
    lhs, rhs = float(np.sum(y * dy)), float(np.sum(x * dx))
    assert abs(lhs - rhs) <= 1e-12 * (np.sum(np.abs(y * dy)) + 1.0)


@pytest.mark.parametrize("X,pad", [((4, 5), 1), ((3, 3), 0), ((2, 4), 2)])
def test_transpose_of_explicit_matrix(X, pad):
    # build the forward map column by column from unit inputs with the loop-nest
    # oracle; its transpose applied to dy is the adjoint, element for element
    C, K, r = 2, 3, 3
    w = _rand((K, C, r, r), 4)
    Y = out_extent(X, pad, r)
    cols = []
    for idx in itertools.product(range(C), *[range(v) for v in X]):
        e = np.zeros((1, C) + X)
        e[(0,) + idx] = 1.0
        cols.append(direct_naive(e, w, pad)[0].ravel())
    A = np.stack(cols, axis=1)                    # [K*prod(Y)] x [C*prod(X)]
    dy = _rand((1, K) + Y, 5)
    want = (A.T @ dy.ravel()).reshape((1, C) + X)
    got, _ = direct_adjoint(dy, w, pad)
    assert np.max(np.abs(got - want)) <= 1e-12


@pytest.mark.parametrize("N,pad", [(1, 1), (2, 0), (2, 1), (2, 2), (3, 1), (3, 0)])
def test_matches_torch_conv_transpose(N, pad):
    r, C, K, n = 3, 3, 5, 2
    Y = (8, 6, 5)[:N]
    w = _rand((K, C) + (r,) * N, 6)
    dy = _rand((n, K) + Y, 7)
    fn = {1: torch.nn.functional.conv_transpose1d, 2: torch.nn.functional.conv_transpose2d,
          3: torch.nn.functional.conv_transpose3d}[N]
    want = fn(torch.from_numpy(dy), torch.from_numpy(w), padding=pad).numpy()
    got, den = direct_adjoint(dy, w, pad)
    assert got.shape == want.shape == (n, C) + in_extent(Y, pad, r)
    assert np.max(np.abs(got - want)) <= 1e-12 * np.max(den)


def test_den_bounds_and_abs_identity():
    # den is the adjoint of |w| applied to |dy|, so it bounds |dx| and equals
    # dx when w and dy are non-negative
    w = np.abs(_rand((4, 3, 3, 3, 3), 8))
    dy = np.abs(_rand((2, 4, 5, 6, 4), 9))
    dx, den = direct_adjoint(dy, w, 1)
    assert np.allclose(dx, den, rtol=1e-13, atol=0)
    w2, dy2 = _rand(w.shape, 10), _rand(dy.shape, 11)
    dx2, den2 = direct_adjoint(dy2, w2, 1)
    assert np.all(np.abs(dx2) <= den2 * (1 + 1e-12))


def test_sampled_matches_full():
    w = _rand((5, 4, 3, 3, 3), 12)
    dy = _rand((2, 5, 6, 5, 7), 13)
    dx, den = direct_adjoint(dy, w, 1)
    rng = np.random.default_rng(14)
    coords = np.stack([rng.integers(0, s, size=300) for s in dx.shape], axis=1)
    coords = np.concatenate([coords, [[0, 0, 0, 0, 0], [1, 3, 5, 4, 6]]])
    v, d = direct_adjoint_sampled(dy, w, 1, coords)
    assert np.allclose(v, dx[tuple(coords.T)], rtol=0, atol=1e-12)
    assert np.allclose(d, den[tuple(coords.T)], rtol=0, atol=1e-12)
