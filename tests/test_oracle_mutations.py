"""Planted mistakes in the oracle (CPU only) must be caught by the pins.

Each case takes a plausible slip (a wrong sign, a dropped term, a transposed
operand, a wrong index or stride) into the oracle's arithmetic and checks that
the exact brute-force comparison against the direct correlation, or the
printed matrices, rejects it.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle.winograd as ow
from golden_io import read_matrices
from oracle.direct import direct_blas, direct_naive
from oracle.toomcook import winograd_matrices


def _exact_case():
    rng = np.random.default_rng(2)
    x = rng.integers(-3, 4, size=(1, 2, 5, 6, 5))
    w = rng.integers(-3, 4, size=(2, 2, 3, 3, 3))
    y_ref, _ = direct_naive(x, w, 1)
    return x, w, y_ref


def _mutated(kind):
    orig = ow.matrices

    def fake(m, r, points=None, exact=False):
        AT, BT, G = orig(m, r, points, exact)
        AT, BT, G = AT.copy(), BT.copy(), G.copy()
        if kind == "sign_G":
            G[1, 1] = -G[1, 1]
        elif kind == "transpose_BT":
            BT = BT.T.copy()
        elif kind == "drop_infinity":
            AT[:, -1] = 0
        elif kind == "scale_AT":
            AT[0, 0] = AT[0, 0] * 2
        elif kind == "swap_rows_G":
            G[[1, 2]] = G[[2, 1]]
        return AT, BT, G
    return fake


@pytest.mark.parametrize("kind", ["sign_G", "transpose_BT", "drop_infinity", "scale_AT",
                                  "swap_rows_G"])
def test_matrix_mutations_caught(monkeypatch, kind):
    x, w, y_ref = _exact_case()
    y_ok = ow.winograd_forward(x, w, 2, 3, pad=1, exact=True)
    assert all(Fraction(float(a)) == b for a, b in zip(y_ref.reshape(-1), y_ok.reshape(-1)))
    monkeypatch.setattr(ow, "matrices", _mutated(kind))
    y_bad = ow.winograd_forward(x, w, 2, 3, pad=1, exact=True)
    assert not all(Fraction(float(a)) == b for a, b in zip(y_ref.reshape(-1), y_bad.reshape(-1)))


def test_generator_sign_rule_pinned_by_printed_matrices():
    points, printed = read_matrices("f23_matrices.txt")
    AT, BT, G = winograd_matrices(2, 3, points)
    flipped = [[-c for c in row] for row in BT]
    assert flipped != printed["BT"]


def test_flipped_kernel_caught_by_library_conv():
    import torch
    rng = np.random.default_rng(9)
    x = rng.standard_normal((1, 2, 5, 5, 5)).astype(np.float32)
    w = rng.standard_normal((2, 2, 3, 3, 3)).astype(np.float32)
    y_flip, _ = direct_blas(x, w[:, :, ::-1, ::-1, ::-1].copy(), 1)
    ref = torch.nn.functional.conv3d(torch.from_numpy(x).double(), torch.from_numpy(w).double(),
                                     padding=1).numpy()
    assert np.abs(y_flip - ref).max() > 1e-3


def test_wrong_tile_stride_caught(monkeypatch):
    """Tiling with stride alpha instead of m misses outputs."""
    x, w, y_ref = _exact_case()
    orig = ow.tile_counts

    def fake(X, pad, m, r):
        Y, T = orig(X, pad, m, r)
        return Y, tuple(max(1, t - 1) for t in T)
    monkeypatch.setattr(ow, "tile_counts", fake)
    y_bad = ow.winograd_forward(x, w, 2, 3, pad=1, exact=True)
    # one tile fewer per axis covers fewer outputs: the result cannot match
    # the direct correlation (a crop too short, or missing values)
    same = y_bad.shape == y_ref.shape and all(
        Fraction(float(a)) == b for a, b in zip(y_ref.reshape(-1), y_bad.reshape(-1)))
    assert not same
    assert y_bad.shape != y_ref.shape
