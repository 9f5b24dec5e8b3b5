"""Pins for the exact transform synthesis in oracle/toomcook.py.

* Printed matrices: F(2,3) of §2.2 and F(4,3) of §3.3, entry for entry.
* Table 1 (§4.2): zero fractions of A, B and the kernel transform, and the
  2-D / 3-D speed-ups, for all five rows.
* The defining identity, exactly in rationals by brute force:
  A^T[(G g) . (B^T d)] = correlation(g, d), and the convolution form of
  eq. (1) equals the polynomial product of §2.1.
* The §2.2 worked example: the element-wise products are the minimal
  algorithm's m1..m4.
"""
import random
from fractions import Fraction

import numpy as np
import pytest

from golden_io import read_kv, read_matrices, read_table1
from oracle import costmodel
from oracle.toomcook import (PAPER_F43_POINTS, default_points, poly_mul,
                             toom_cook_convolution, winograd_matrices)


def _mat(M):
    return [[Fraction(c) for c in row] for row in M]


@pytest.mark.parametrize("fixture,m", [("f23_matrices.txt", 2), ("f43_matrices.txt", 4)])
def test_printed_matrices(fixture, m):
    points, printed = read_matrices(fixture)
    AT, BT, G = winograd_matrices(m, 3, points)
    assert _mat(AT) == printed["AT"]
    assert _mat(BT) == printed["BT"]
    assert _mat(G) == printed["G"]


def test_paper_f43_points_constant_matches_fixture():
    points, _ = read_matrices("f43_matrices.txt")
    assert list(PAPER_F43_POINTS) == points


def _zero_frac(M):
    n = sum(len(r) for r in M)
    return sum(1 for r in M for c in r if c == 0) / n


def test_table1():
    half = Fraction(1, 2)
    eight = (0, 1, -1, 2, -2, half, -half)
    for key, row in read_table1().items():
        S, Gk, D = row["S"], row["G"], row["D"]
        assert S + Gk - 1 == D
        pts = (0, 1, -1) if D == 4 else eight
        AT, BT, G = winograd_matrices(S, Gk, pts)
        assert round(_zero_frac(AT), 2) == row["zA"], key
        assert round(_zero_frac(BT), 2) == row["zB"], key
        assert round(_zero_frac(G), 2) == row["zC"], key
        # printed to two decimals, rounding half up (15.625 -> 15.63)
        assert abs(costmodel.ideal_speedup(S, Gk, 2) - row["su2"]) <= 0.005 + 1e-12, key
        assert abs(costmodel.ideal_speedup(S, Gk, 3) - row["su3"]) <= 0.005 + 1e-12, key


def _corr(g, d, m):
    return [sum(g[k] * d[i + k] for k in range(len(g))) for i in range(m)]


def _apply(M, v):
    return [sum(a * b for a, b in zip(row, v)) for row in M]


CASES = [
    (2, 3, (0, 1, -1)), (4, 3, (0, 1, -1, 2, -2)), (4, 3, PAPER_F43_POINTS),
    (2, 2, (0, 1)), (3, 2, (0, 1, -1)), (3, 3, (0, 1, -1, 2)),
    (5, 4, (0, 1, -1, 2, -2, Fraction(1, 2), Fraction(-1, 2))),
    (2, 5, (0, 1, -1, 2, -2)), (1, 3, (0, 1)), (2, 3, (1, 2, 3)),
    (4, 3, (0, -1, 1, Fraction(1, 2), -2)),
]


@pytest.mark.parametrize("m,r,points", CASES)
def test_correlation_identity_bruteforce(m, r, points):
    rng = random.Random(1000 * m + r)
    AT, BT, G = winograd_matrices(m, r, points)
    alpha = m + r - 1
    assert len(AT) == m and len(AT[0]) == alpha
    assert len(BT) == alpha and len(BT[0]) == alpha
    assert len(G) == alpha and len(G[0]) == r
    for _ in range(60):
        g = [Fraction(rng.randint(-9, 9)) for _ in range(r)]
        d = [Fraction(rng.randint(-9, 9)) for _ in range(alpha)]
        prod = [a * b for a, b in zip(_apply(G, g), _apply(BT, d))]
        assert _apply(AT, prod) == _corr(g, d, m)
    # Unit inputs make every entry of the bilinear form visible.
    for k in range(r):
        for j in range(alpha):
            g = [Fraction(int(i == k)) for i in range(r)]
            d = [Fraction(int(i == j)) for i in range(alpha)]
            prod = [a * b for a, b in zip(_apply(G, g), _apply(BT, d))]
            assert _apply(AT, prod) == _corr(g, d, m)


@pytest.mark.parametrize("m,r,points", CASES[:6])
def test_convolution_form_is_polynomial_product(m, r, points):
    """Eq. (1) s = A[(C g) . (B d)] reproduces s(x) = g(x) d(x) (§2.1)."""
    A_cv, B, C = toom_cook_convolution(m, r, points)
    rng = random.Random(7)
    for _ in range(30):
        g = [Fraction(rng.randint(-5, 5)) for _ in range(r)]
        u = [Fraction(rng.randint(-5, 5)) for _ in range(m)]
        s = _apply(A_cv, [a * b for a, b in zip(_apply(C, g), _apply(B, u))])
        want = poly_mul(g, u)
        want = want + [Fraction(0)] * (len(s) - len(want))
        assert s == want


def test_hand_example_minimal_f23():
    ex = read_kv("f23_hand_example.txt")
    AT, BT, G = winograd_matrices(2, 3, default_points(2, 3))
    prod = [a * b for a, b in zip(_apply(G, ex["g"]), _apply(BT, ex["d"]))]
    assert prod == ex["m"]
    assert _apply(AT, prod) == ex["s"]
    assert _corr(ex["g"], ex["d"], 2) == ex["s"]


def test_rejects_bad_points():
    with pytest.raises(ValueError):
        winograd_matrices(2, 3, (0, 1, 1))
    with pytest.raises(ValueError):
        winograd_matrices(2, 3, (0, 1))
    with pytest.raises(ValueError):
        winograd_matrices(4, 3, (0, 1, -1, 2))


def test_float_rounding_is_single_rounding():
    AT, BT, G = winograd_matrices(4, 3, PAPER_F43_POINTS)
    for M in (AT, BT, G):
        for row in M:
            for c in row:
                f = float(c)
                # nearest double: the exact rational lies within half an ulp
                assert abs(Fraction(f) - c) <= Fraction(np.spacing(abs(f))) / 2
