"""Pins for the multiplication counts in oracle/costmodel.py (§3.2-§3.3, Table 1)."""
import pytest

from oracle import costmodel


def test_f23_explicit_count():
    # §3.3: 4 products + 16 data-transform + 8 inverse-transform multiplications.
    assert costmodel.explicit_1d_mults(2, 3) == 28


@pytest.mark.parametrize("M", [1, 8, 100])
def test_f23_layer_count(M):
    # §3.3: 4M^2 + 24M with transformed kernels cached.
    assert costmodel.layer_1d_mults(2, 3, M) == 4 * M * M + 24 * M


def test_c3d_reduction_quotes():
    # §3.3: the F(4,3) C3D matrices cap the speed-up at 8; with 100 channels and
    # 100 kernels the reduction is greater than 6-fold, about triple the margin
    # available with 10 of each.
    assert costmodel.ideal_speedup(4, 3, 3) == pytest.approx(8.0)
    d100, f100 = costmodel.c3d_tile_mults(4, 3, 100, 100)
    d10, f10 = costmodel.c3d_tile_mults(4, 3, 10, 10)
    r100, r10 = d100 / f100, d10 / f10
    assert r100 > 6.0
    assert 2.5 < r100 / r10 < 3.5
    assert r100 < 8.0


def test_speedups_of_workload_tiles():
    assert costmodel.ideal_speedup(2, 3, 3) == pytest.approx(3.375)
    assert costmodel.ideal_speedup(4, 3, 2) == pytest.approx(4.0)
