"""Pins of the weight-gradient oracle (oracle/wgrad.py) against facts outside it."""
import itertools

import numpy as np
import pytest
import torch

from oracle.direct import direct_blas, direct_naive, out_extent
from oracle.wgrad import direct_wgrad


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


@pytest.mark.parametrize("N,r,pad", [(1, 3, 1), (2, 3, 1), (2, 3, 0), (3, 3, 1), (3, 3, 2), (2, 4, 1),
                                     (2, 2, 0), (2, 3, 4)])
def test_inner_product_identity(N, r, pad):
    # y is linear in w: <dy, corr(x, w)> = <w, dw> for every w
    X = (8, 7, 6)[:N]
    C, K, n = 3, 4, 2
    x = _rand((n, C) + X, 1)
    w = _rand((K, C) + (r,) * N, 2)
    y, _ = direct_blas(x, w, pad, with_den=False)
    dy = _rand(y.shape, 3)
    dw, _ = direct_wgrad(x, dy, r, pad)
    lhs, rhs = float(np.sum(y * dy)), float(np.sum(w * dw))
    assert abs(lhs - rhs) <= 1e-12 * (np.sum(np.abs(y * dy)) + 1.0)


def test_unit_kernel_responses():
    # dw[k][c][p] = <dy, forward response to the unit kernel at (k, c, p)>,
    # through the loop-nest oracle
    C, K, r, pad, X = 2, 2, 3, 1, (4, 5)
    x = _rand((2, C) + X, 4)
    dy = _rand((2, K) + out_extent(X, pad, r), 5)
    want = np.zeros((K, C, r, r))
    for k, c, p0, p1 in itertools.product(range(K), range(C), range(r), range(r)):
        e = np.zeros((K, C, r, r))
        e[k, c, p0, p1] = 1.0
        want[k, c, p0, p1] = np.sum(direct_naive(x, e, pad)[0] * dy)
    got, _ = direct_wgrad(x, dy, r, pad)
    assert np.max(np.abs(got - want)) <= 1e-12


@pytest.mark.parametrize("N,pad", [(2, 0), (2, 1), (3, 1), (3, 0)])
def test_matches_torch_weight_grad(N, pad):
    r, C, K, n = 3, 3, 5, 2
    X = (9, 7, 6)[:N]
    x = _rand((n, C) + X, 6)
    dy = _rand((n, K) + out_extent(X, pad, r), 7)
    fn = {2: torch.nn.grad.conv2d_weight, 3: torch.nn.grad.conv3d_weight}[N]
    want = fn(torch.from_numpy(x), (K, C) + (r,) * N, torch.from_numpy(dy), padding=pad).numpy()
    got, den = direct_wgrad(x, dy, r, pad)
    assert np.max(np.abs(got - want)) <= 1e-12 * np.max(den)


def test_den_bounds():
    x, dy = _rand((2, 3, 6, 5, 4), 8), _rand((2, 4, 6, 5, 4), 9)
    dw, den = direct_wgrad(x, dy, 3, 1)
    assert np.all(np.abs(dw) <= den * (1 + 1e-12))
    dwa, dena = direct_wgrad(np.abs(x), np.abs(dy), 3, 1)
    assert np.allclose(dwa, dena, rtol=1e-13, atol=0)
