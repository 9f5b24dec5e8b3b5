"""Pins for the reference Winograd (oracle/winograd.py).

* Exact agreement with the direct correlation on small integer inputs, by
  brute force in rationals: N = 1, 2, 3, every supported (m, r) and point
  set, ragged tiles, pad 0 and 1, several channels and kernels.
* fp64 agreement with the direct correlation on random inputs.
* Separability (eq. 3 and 4): the N-D data transform equals the Kronecker
  product of the 1-D transform applied to the vectorised tile, and every axis
  order gives the same tensor.
* The 2-D special case of §3.2: A[(C g C^T) . (B d B^T)]A^T in matrix form.
* The §2.2 worked example.
* Exact invariants of a correlation that tiling and stitching must keep:
  translation by shifts that are not multiples of m, linearity, batch
  independence, and a one-hot kernel selecting the input window (no flip).
"""
import itertools
import random
from fractions import Fraction

import numpy as np
import pytest

from golden_io import read_kv
from oracle.direct import direct_blas, direct_naive
from oracle.metric import normalised_error
from oracle.toomcook import PAPER_F43_POINTS
from oracle.winograd import matrices, mode_products, winograd_forward

EXACT_CASES = [
    # N, m, r, points, n, C, K, X, pad
    (1, 2, 3, None, 2, 2, 3, (9,), 0),
    (1, 4, 3, None, 1, 3, 2, (11,), 1),
    (1, 3, 2, None, 1, 2, 2, (8,), 0),
    (2, 2, 3, None, 1, 2, 3, (5, 6), 1),
    (2, 4, 3, None, 2, 2, 2, (7, 5), 1),
    (2, 4, 3, PAPER_F43_POINTS, 1, 2, 2, (6, 7), 0),
    (2, 2, 2, None, 1, 3, 2, (5, 4), 0),
    (3, 2, 3, None, 1, 2, 2, (5, 4, 6), 1),
    (3, 2, 3, None, 2, 3, 2, (4, 4, 4), 0),
    (3, 4, 3, None, 1, 2, 2, (5, 6, 4), 1),
    (3, 4, 3, PAPER_F43_POINTS, 1, 2, 2, (6, 6, 6), 0),
    (1, 5, 4, None, 1, 2, 2, (17,), 1),
    (2, 5, 4, None, 1, 2, 2, (12, 9), 0),
    (2, 5, 4, None, 1, 1, 2, (8, 13), 1),
    (2, 4, 5, None, 1, 2, 2, (11, 12), 0),
    (2, 3, 6, None, 1, 2, 1, (13, 10), 1),
    (2, 3, 2, None, 2, 2, 2, (7, 8), 1),
    # Table 1's sizes in 3-D (alpha = 4 and 8): one or two ragged tiles per axis
    (3, 3, 2, None, 1, 2, 2, (5, 4, 6), 1),
    (3, 5, 4, None, 1, 1, 2, (8, 6, 9), 0),
    (3, 4, 5, None, 1, 2, 1, (8, 9, 6), 1),
    (3, 3, 6, None, 1, 1, 1, (9, 8, 7), 1),
]


@pytest.mark.parametrize("N,m,r,points,n,C,K,X,pad", EXACT_CASES)
def test_exact_equals_direct(N, m, r, points, n, C, K, X, pad):
    rng = np.random.default_rng(abs(hash((N, m, r, X))) % 2**32)
    x = rng.integers(-3, 4, size=(n, C) + X)
    w = rng.integers(-3, 4, size=(K, C) + (r,) * N)
    y_ref, _ = direct_naive(x, w, pad)
    y = winograd_forward(x, w, m, r, pad=pad, points=points, exact=True)
    assert y.shape == y_ref.shape
    assert all(isinstance(v, Fraction) for v in y.reshape(-1)[:5])
    assert all(Fraction(float(a)) == b for a, b in zip(y_ref.reshape(-1), y.reshape(-1)))
    yr = winograd_forward(x, w, m, r, pad=pad, points=points, exact=True, relu=True)
    assert all(Fraction(float(max(a, 0))) == b for a, b in zip(y_ref.reshape(-1), yr.reshape(-1)))


@pytest.mark.parametrize("N,m,r,X,pad", [(3, 2, 3, (7, 9, 8), 1), (2, 4, 3, (13, 10), 1),
                                          (3, 4, 3, (9, 7, 10), 1), (1, 4, 3, (30,), 0)])
def test_fp64_close_to_direct(N, m, r, X, pad):
    rng = np.random.default_rng(11)
    x = rng.standard_normal((2, 5) + X).astype(np.float32)
    w = rng.standard_normal((3, 5) + (r,) * N).astype(np.float32)
    y_ref, den = direct_blas(x, w, pad)
    y = winograd_forward(x, w, m, r, pad=pad)
    assert normalised_error(y, y_ref, den)["max"] < 1e-12


def _kron_all(M, N):
    K = np.array([[1]], dtype=object)
    for _ in range(N):
        K = np.kron(K, M)
    return K


@pytest.mark.parametrize("N,m,r", [(2, 2, 3), (3, 2, 3), (2, 4, 3), (3, 4, 3), (2, 5, 4)])
def test_separability(N, m, r):
    AT, BT, G = matrices(m, r, exact=True)
    alpha = m + r - 1
    rng = random.Random(N * 31 + m)
    d = np.array([Fraction(rng.randint(-4, 4)) for _ in range(alpha ** N)],
                 dtype=object).reshape((alpha,) * N)
    ref = _kron_all(BT, N).dot(d.reshape(-1)).reshape((alpha,) * N)
    for order in itertools.permutations(range(N)):
        got = mode_products(d, [BT] * N, list(order))
        assert (got == ref).all()
    g = np.array([Fraction(rng.randint(-4, 4)) for _ in range(r ** N)],
                 dtype=object).reshape((r,) * N)
    refg = _kron_all(G, N).dot(g.reshape(-1)).reshape((alpha,) * N)
    for order in itertools.permutations(range(N)):
        assert (mode_products(g, [G] * N, list(order)) == refg).all()


def test_2d_lavin_form():
    AT, BT, G = matrices(4, 3, exact=True)
    rng = random.Random(5)
    d = np.array([[Fraction(rng.randint(-4, 4)) for _ in range(6)] for _ in range(6)], dtype=object)
    g = np.array([[Fraction(rng.randint(-4, 4)) for _ in range(3)] for _ in range(3)], dtype=object)
    # The paper's A, B, C are A^T, B^T, G here: S = A[(C g C^T) . (B d B^T)]A^T.
    S = AT.dot((G.dot(g).dot(G.T)) * (BT.dot(d).dot(BT.T))).dot(AT.T)
    y = winograd_forward(d.reshape(1, 1, 6, 6), g.reshape(1, 1, 3, 3), 4, 3, exact=True)
    assert (y.reshape(4, 4) == S).all()
    y2, _ = direct_naive(d.astype(float).reshape(1, 1, 6, 6), g.astype(float).reshape(1, 1, 3, 3))
    assert (S.astype(float) == y2.reshape(4, 4)).all()


def test_hand_example():
    ex = read_kv("f23_hand_example.txt")
    d = np.array(ex["d"], dtype=object).reshape(1, 1, 4)
    g = np.array(ex["g"], dtype=object).reshape(1, 1, 3)
    y = winograd_forward(d, g, 2, 3, exact=True)
    assert list(y.reshape(-1)) == ex["s"]


def test_output_extent_must_be_positive():
    with pytest.raises(ValueError):
        winograd_forward(np.zeros((1, 1, 2, 2)), np.zeros((1, 1, 3, 3)), 2, 3)


def test_nonfinite_input_poisons_tile():
    """A NaN in x poisons every output of each tile whose window holds it; the
    direct correlation only poisons outputs whose receptive field holds it.
    Finite inputs are required."""
    x = np.ones((1, 1, 8, 8), np.float32)
    x[0, 0, 4, 4] = np.nan
    w = np.ones((1, 1, 3, 3), np.float32)
    y = winograd_forward(x, w, 2, 3)
    yd, _ = direct_blas(x, w, 0)
    assert np.isnan(y).sum() >= np.isnan(yd).sum()


# ---- invariants of the correlation that the Winograd path must keep exactly
def _exact(x, w, m, pad=0):
    return winograd_forward(x, w, m, 3, pad=pad, exact=True)


@pytest.mark.parametrize("N,m,axis,s", [(2, 2, 1, 1), (2, 4, 0, 3), (3, 2, 2, 1), (3, 4, 0, 1)])
def test_translation_equivariance(N, m, axis, s):
    """Shifting the input by s along an axis shifts the valid output by s:
    the tile grid (stride m) must not leak into the result."""
    rng = np.random.default_rng(7 + N + m + s)
    X = (7, 6, 5)[:N] if N == 3 else (9, 8)
    x = rng.integers(-3, 4, size=(1, 2) + X)
    w = rng.integers(-3, 4, size=(2, 2) + (3,) * N)
    xs = np.zeros_like(x)
    src = [slice(None)] * (N + 2)
    dst = [slice(None)] * (N + 2)
    src[2 + axis] = slice(0, X[axis] - s)
    dst[2 + axis] = slice(s, X[axis])
    xs[tuple(dst)] = x[tuple(src)]
    y, ys = _exact(x, w, m), _exact(xs, w, m)
    keep_y = [slice(None)] * (N + 2)
    keep_ys = [slice(None)] * (N + 2)
    Y = y.shape[2 + axis]
    keep_y[2 + axis] = slice(0, Y - s)
    keep_ys[2 + axis] = slice(s, Y)
    assert np.array_equal(ys[tuple(keep_ys)], y[tuple(keep_y)])


def test_linearity_exact():
    rng = np.random.default_rng(3)
    x1 = rng.integers(-3, 4, size=(1, 2, 6, 5, 7))
    x2 = rng.integers(-3, 4, size=(1, 2, 6, 5, 7))
    w = rng.integers(-3, 4, size=(2, 2, 3, 3, 3))
    lhs = _exact(2 * x1 - 3 * x2, w, 2, pad=1)
    rhs = 2 * _exact(x1, w, 2, pad=1) - 3 * _exact(x2, w, 2, pad=1)
    assert np.array_equal(lhs, rhs)


def test_batch_independence_exact():
    rng = np.random.default_rng(4)
    x = rng.integers(-3, 4, size=(2, 2, 5, 6, 5))
    w = rng.integers(-3, 4, size=(3, 2, 3, 3, 3))
    both = _exact(x, w, 4, pad=1)
    assert np.array_equal(both[:1], _exact(x[:1], w, 4, pad=1))
    assert np.array_equal(both[1:], _exact(x[1:], w, 4, pad=1))


@pytest.mark.parametrize("p", [(0, 0, 0), (2, 1, 0), (1, 2, 2)])
def test_one_hot_kernel_selects_input(p):
    """A kernel with a single 1 at offset p returns the input window at p: no flip."""
    rng = np.random.default_rng(5)
    x = rng.integers(-5, 6, size=(1, 1, 6, 7, 5))
    w = np.zeros((1, 1, 3, 3, 3), dtype=np.int64)
    w[(0, 0) + p] = 1
    y = _exact(x, w, 2)
    Y = y.shape[2:]
    want = x[0, 0, p[0]:p[0] + Y[0], p[1]:p[1] + Y[1], p[2]:p[2] + Y[2]]
    assert np.array_equal(y[0, 0], want)


# ---- per-axis transforms (eq. 4 with its own C_n, B_n, A_n on each axis)
ANISO_EXACT = [
    # N, m per axis, r, n, C, K, X, pad
    (3, (2, 4, 4), 3, 1, 2, 2, (5, 9, 7), 1),
    (3, (4, 2, 2), 3, 1, 2, 3, (7, 4, 5), 1),
    (3, (2, 4, 4), 3, 2, 2, 2, (3, 6, 6), 0),
    (3, (4, 2, 2), 3, 1, 3, 2, (6, 5, 3), 0),
    (3, (2, 4, 2), 3, 1, 2, 2, (4, 7, 5), 1),
    (2, (2, 4), 3, 1, 2, 2, (7, 9), 1),
    (2, (4, 2), 3, 2, 2, 3, (6, 5), 0),
    (2, (3, 5), 4, 1, 2, 2, (9, 11), 1),
]


@pytest.mark.parametrize("N,ms,r,n,C,K,X,pad", ANISO_EXACT)
def test_anisotropic_exact_equals_direct(N, ms, r, n, C, K, X, pad):
    """Mixed per-axis tiles reach the direct correlation exactly (rationals):
    ragged tiles on every axis, pad 0 and 1."""
    rng = np.random.default_rng(abs(hash((N, ms, X))) % 2**32)
    x = rng.integers(-3, 4, size=(n, C) + X)
    w = rng.integers(-3, 4, size=(K, C) + (r,) * N)
    y_ref, _ = direct_naive(x, w, pad)
    y = winograd_forward(x, w, ms, r, pad=pad, exact=True)
    assert y.shape == y_ref.shape
    assert all(Fraction(float(a)) == b for a, b in zip(y_ref.reshape(-1), y.reshape(-1)))


def test_anisotropic_separability():
    """The N-D data and kernel transforms with per-axis matrices equal the
    Kronecker product of the per-axis 1-D transforms applied to the
    vectorised tile, in any axis order (exact)."""
    ms, r = (2, 4, 4), 3
    mats = [matrices(mi, r, exact=True) for mi in ms]
    alphas = tuple(mi + r - 1 for mi in ms)
    rng = random.Random(17)
    d = np.array([Fraction(rng.randint(-4, 4)) for _ in range(int(np.prod(alphas)))],
                 dtype=object).reshape(alphas)
    kB = np.kron(np.kron(mats[0][1], mats[1][1]), mats[2][1])
    ref = kB.dot(d.reshape(-1)).reshape(alphas)
    for order in itertools.permutations(range(3)):
        got = mode_products(d, [mats[a][1] for a in order], list(order))
        assert (got == ref).all()
    g = np.array([Fraction(rng.randint(-4, 4)) for _ in range(r ** 3)], dtype=object).reshape((r,) * 3)
    kG = np.kron(np.kron(mats[0][2], mats[1][2]), mats[2][2])
    refg = kG.dot(g.reshape(-1)).reshape(alphas)
    assert (mode_products(g, [mats[a][2] for a in range(3)], [0, 1, 2]) == refg).all()


def test_anisotropic_axis_mistakes_caught():
    """Planted mistakes in the per-axis matrices: the first axis's B^T applied
    along the second (sizes 4 and 6 clash), and a dropped CRT factor in one
    axis's G only (the result is no longer the correlation)."""
    import oracle.winograd as ow
    orig = ow._axis_matrices
    x = np.random.default_rng(3).integers(-3, 4, size=(1, 2, 5, 7, 6))
    w = np.random.default_rng(4).integers(-3, 4, size=(2, 2, 3, 3, 3))

    def swapped(m, r, N, points, exact):
        mats = orig(m, r, N, points, exact)
        (A0, B0, G0), (A1, B1, G1) = mats[0], mats[1]
        return [(A0, B1, G0), (A1, B0, G1)] + mats[2:]
    ow._axis_matrices = swapped
    try:
        with pytest.raises(ValueError):
            ow.winograd_forward(x, w, (2, 4, 4), 3, pad=1, exact=True)
    finally:
        ow._axis_matrices = orig

    def scaled(m, r, N, points, exact):
        mats = orig(m, r, N, points, exact)
        A0, B0, G0 = mats[0]
        return [(A0, B0, G0 * 2)] + mats[1:]
    y_ref, _ = direct_naive(x, w, 1)
    good = ow.winograd_forward(x, w, (2, 4, 4), 3, pad=1, exact=True)
    assert all(Fraction(float(a)) == b for a, b in zip(y_ref.reshape(-1), good.reshape(-1)))
    ow._axis_matrices = scaled
    try:
        bad = ow.winograd_forward(x, w, (2, 4, 4), 3, pad=1, exact=True)
    finally:
        ow._axis_matrices = orig
    assert not all(Fraction(float(a)) == b for a, b in zip(y_ref.reshape(-1), bad.reshape(-1)))


def test_anisotropic_points_rejected():
    with pytest.raises(ValueError):
        winograd_forward(np.zeros((1, 1, 5, 5, 5)), np.zeros((1, 1, 3, 3, 3)), (2, 4, 4), 3,
                         points=(0, 1, -1))
