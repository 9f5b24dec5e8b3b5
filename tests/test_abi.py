"""Host-side checks of the C ABI (no GPU needed: no device work is launched).

* libwino.so loads and exports every function include/wino.h declares.
* wino_plan validates its arguments and reports sizes and output extents.
* The C++ transform synthesis equals the oracle's exact synthesis rounded
  once to double, bit for bit (default points, the paper's F(4,3) points and
  other caller-chosen sets).
* Device entry points reject bad pointers and short workspaces synchronously,
  before any launch.
"""
import ctypes
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle.toomcook import PAPER_F43_POINTS, default_points, winograd_matrices

wino = pytest.importorskip("paper_1611_06565_amd.wino")


@pytest.fixture(scope="module")
def L():
    return wino.lib()


def test_exports_every_header_symbol(L):
    names = wino.describe_header_symbols()
    assert len(names) >= 13
    for n in names:
        assert hasattr(L, n), n


def test_status_strings(L):
    assert L.wino_status_string(0) == b"ok"
    assert L.wino_status_string(-3) == b"workspace too small"


def _plan_status(L, N, m, r, C, K, dims, pad=None, points=None, flags=0, slope=0.0):
    opts = wino._Opts()
    if pad is not None:
        for i, p in enumerate(pad):
            opts.pad[i] = p
    keep = None
    if points is not None:
        keep = (ctypes.c_double * len(points))(*points)
        opts.points = ctypes.cast(keep, ctypes.POINTER(ctypes.c_double))
        opts.n_points = len(points)
    opts.flags = flags
    opts.slope = slope
    arr = (ctypes.c_int64 * len(dims))(*dims)
    h = ctypes.c_void_p()
    st = L.wino_plan(N, m, r, C, K, arr, ctypes.byref(opts), ctypes.byref(h))
    if st == 0:
        L.wino_destroy(h)
    return st


def test_plan_validation(L):
    ok = _plan_status(L, 3, 2, 3, 4, 4, [1, 8, 8, 8])
    assert ok == 0
    assert _plan_status(L, 4, 2, 3, 4, 4, [1, 8, 8, 8, 8]) == -1      # N out of range
    assert _plan_status(L, 3, 3, 3, 4, 4, [1, 8, 8, 8]) == -2         # no kernel for m = 3
    assert _plan_status(L, 3, 2, 5, 4, 4, [1, 8, 8, 8]) == -2         # r = 5
    # Table 1's sizes in 3-D
    for m, r in ((3, 2), (5, 4), (4, 5), (3, 6)):
        assert _plan_status(L, 3, m, r, 4, 4, [1, 9, 9, 9]) == 0, (m, r)
    assert _plan_status(L, 3, 6, 3, 4, 4, [1, 9, 9, 9]) == -2         # alpha = 8, no kernel for m = 6
    assert _plan_status(L, 3, 2, 3, 0, 4, [1, 8, 8, 8]) == -1         # C = 0
    assert _plan_status(L, 3, 2, 3, 4, 0, [1, 8, 8, 8]) == -1         # K = 0
    assert _plan_status(L, 3, 2, 3, 4, 4, [0, 8, 8, 8]) == -1         # batch 0
    assert _plan_status(L, 3, 2, 3, 4, 4, [1, 2, 8, 8]) == -1         # Y < 1 unpadded
    assert _plan_status(L, 3, 2, 3, 4, 4, [1, 2, 8, 8], pad=[1, 0, 0]) == 0
    assert _plan_status(L, 3, 2, 3, 4, 4, [1, 8, 8, 8], pad=[-1, 0, 0]) == -1
    assert _plan_status(L, 3, 2, 3, 4, 4, [1, 8, 8, 8], points=[0, 1, 1]) == -1   # duplicate
    assert _plan_status(L, 3, 2, 3, 4, 4, [1, 8, 8, 8], points=[0, 1]) == -1      # count
    assert _plan_status(L, 3, 2, 3, 4, 4, [1, 8, 8, 8], points=[0, 1, math.nan]) == -1
    assert _plan_status(L, 3, 2, 3, 4, 4, [1, 8, 8, 8], points=[0, 1, math.pi]) == -1
    assert _plan_status(L, 3, 2, 3, 4, 4, [1, 8, 8, 8], flags=16) == -1      # unknown flag
    assert _plan_status(L, 3, 4, 3, 4, 4, [1, 8, 8, 8], flags=8) == 0        # WINO_NO_FUSE
    assert _plan_status(L, 3, 2, 3, 4, 4, [1, 8, 8, 8], flags=3) == 0
    assert _plan_status(L, 3, 2, 3, 4, 4, [1, 8, 8, 8], flags=4) == 0        # leaky ReLU, slope 0
    assert _plan_status(L, 3, 2, 3, 4, 4, [1, 8, 8, 8], flags=5) == -1       # two activations
    assert _plan_status(L, 3, 2, 3, 4, 4, [1, 8, 8, 8], flags=4, slope=math.nan) == -1
    assert _plan_status(L, 3, 2, 3, 4, 4, [1, 8, 8, 8], flags=4, slope=math.inf) == -1
    assert _plan_status(L, 3, 2, 3, 4, 4, [1, 8, 8, 8], flags=6, slope=0.1) == 0
    h = ctypes.c_void_p()
    assert L.wino_plan(3, 2, 3, 4, 4, None, None, ctypes.byref(h)) == -1


def test_sizes_and_dims():
    p = wino.Plan(3, 2, 3, 64, 128, [8, 16, 56, 56], pad=1)
    d = p.desc
    assert d["tiles"] == [8, 28, 28] and d["T"] == 8 * 8 * 28 * 28
    assert d["n_xi"] == 64 and d["alpha"] == 4
    assert p.filter_bytes == 4 * 64 * d["C_pad"] * d["K_pad"]
    assert p.workspace_bytes == 4 * 64 * d["C_pad"] * d["T_pad"]
    assert d["gemm_parts"] == 1          # 3136 product blocks: no pass split
    assert p.output_shape == (8, 128, 16, 56, 56)
    q = wino.Plan(2, 4, 3, 3, 5, [2, 9, 10], pad=0)
    assert q.output_shape == (2, 5, 7, 8)
    assert q.desc["tiles"][:2] == [2, 2]
    assert q.desc["T_pad"] % q.desc["block_tiles"] == 0
    assert q.desc["K_pad"] % q.desc["block_kernels"] == 0
    assert q.desc["C_pad"] >= 3


def _oracle_f64(m, r, pts):
    AT, BT, G = winograd_matrices(m, r, pts)
    f = lambda M: np.array([[float(c) for c in row] for row in M])
    return f(AT), f(BT), f(G)


@pytest.mark.parametrize("N,m,pts", [
    (3, 2, None), (2, 2, None), (3, 4, None), (2, 4, None),
    (3, 4, PAPER_F43_POINTS), (2, 4, PAPER_F43_POINTS),
    (3, 2, (1, 2, 3)), (2, 4, (0, -1, 1, 0.5, -2)), (3, 2, (0, 0.5, -0.5)),
])
def test_matrices_bitwise_equal_oracle(N, m, pts):
    plan = wino.Plan(N, m, 3, 2, 2, [1] + [9] * N, pad=1, points=pts)
    AT, BT, G = plan.matrices()
    oAT, oBT, oG = _oracle_f64(m, 3, pts if pts is not None else default_points(m, 3))
    for a, b in ((AT, oAT), (BT, oBT), (G, oG)):
        assert a.shape == b.shape
        assert np.array_equal(a.view(np.uint64), b.view(np.uint64))
    assert plan.desc["default_points"] == (1 if pts is None else 0)


@pytest.mark.parametrize("m,r,pts", [
    (5, 4, None), (5, 4, (0, 1, -1, 2, -2, 0.5, -0.5)), (5, 4, (0, 1, -1, 3, -3, 2, -2)),
    (4, 5, None), (3, 6, None), (3, 2, None), (3, 2, (0, 2, -1)),
])
def test_matrices_bitwise_equal_oracle_2d_sizes(m, r, pts):
    """The other 2-D sizes of Table 1: compiled default constants and caller points."""
    plan = wino.Plan(2, m, r, 2, 2, [1, 12, 12], pad=0, points=pts)
    AT, BT, G = plan.matrices()
    oAT, oBT, oG = _oracle_f64(m, r, pts if pts is not None else default_points(m, r))
    for a, b in ((AT, oAT), (BT, oBT), (G, oG)):
        assert a.shape == b.shape
        assert np.array_equal(a.view(np.uint64), b.view(np.uint64))
    assert plan.desc["default_points"] == (1 if pts is None or tuple(pts) == tuple(default_points(m, r)) else 0)


def test_explicit_default_points_use_compiled_constants():
    plan = wino.Plan(3, 2, 3, 2, 2, [1, 8, 8, 8], points=(0, 1, -1))
    assert plan.desc["default_points"] == 1


def test_device_calls_reject_bad_arguments(L):
    # Every call below must be rejected on the host before any launch: only
    # NULL or misaligned pointers, or short workspaces, are passed.
    p = wino.Plan(2, 4, 3, 4, 4, [1, 8, 8])
    need = p.workspace_bytes
    vp = ctypes.c_void_p
    assert L.wino_transform_filter(p.handle, None, vp(4096), None) == -1
    assert L.wino_transform_filter(p.handle, vp(4096 + 4), vp(4096), None) == -1
    assert L.wino_transform_input(p.handle, vp(4096), vp(8192), need - 4, None) == -3
    assert L.wino_gemm_inverse(p.handle, vp(4096), need - 4, vp(8192), vp(16384), None) == -3
    assert L.wino_forward(p.handle, vp(4096), vp(8192), vp(16384), vp(32768), 0, None) == -3
    assert L.wino_forward(p.handle, vp(4096), vp(8192), vp(16384), None, need, None) == -1
    f = wino.Plan(3, 2, 3, 4, 4, [1, 8, 8, 8])
    assert f.workspace_bytes > 0
    assert L.wino_forward(f.handle, None, vp(8192), vp(16384), vp(32768), 1 << 30, None) == -1
    assert L.wino_forward(f.handle, vp(4096 + 4), vp(8192), vp(16384), vp(32768), 1 << 30, None) == -1
    assert L.wino_forward(f.handle, vp(4096), vp(8192), vp(16384 + 8), vp(32768), 1 << 30, None) == -1
    # the bias variants: a misaligned bias, then the checks of the plain calls
    assert L.wino_forward_ex(f.handle, vp(4096), vp(8192), vp(512 + 2), vp(16384), vp(32768), 1 << 30,
                             None) == -1
    assert L.wino_gemm_inverse_ex(f.handle, vp(4096), 1 << 30, vp(8192), vp(512 + 1), vp(16384), None) == -1
    assert L.wino_forward_ex(f.handle, vp(4096), vp(8192), vp(512), vp(16384), vp(32768), 0, None) == -3
    assert L.wino_gemm_inverse_ex(p.handle, vp(4096), need - 4, vp(8192), None, vp(16384), None) == -3
    assert L.wino_forward_ex(f.handle, None, vp(8192), None, vp(16384), vp(32768), 1 << 30, None) == -1
    dims = (ctypes.c_int64 * 4)(1, 4, 4, 4)
    win = (ctypes.c_int32 * 3)(2, 2, 8)
    assert L.wino_maxpool3d(dims, win, vp(4096), vp(8192), None) == -1   # 4 // 8 == 0


def test_forward_pool_rejects_before_launch(L):
    """wino_forward_pool's refusals, all decided on the host: windows other
    than (1, 2, 2) and (2, 2, 2) (F(2^3): (2, 2, 2) only), sizes whose
    product has no pooled epilogue, pooled extents of 0, bad pointers and a
    missing workspace."""
    vp = ctypes.c_void_p
    W = lambda *w: (ctypes.c_int32 * 3)(*w)
    fused = wino.Plan(3, 4, 3, 4, 16, [1, 8, 8, 8], pad=1)          # F(4^3), K <= 64: fused
    two = wino.Plan(3, 4, 3, 4, 80, [1, 8, 8, 8], pad=1)            # K > 64: two stages
    m2 = wino.Plan(3, 2, 3, 4, 16, [1, 8, 8, 8], pad=1)             # F(2^3): window (2, 2, 2) only
    m32 = wino.Plan(3, 3, 2, 4, 16, [1, 8, 8, 8], pad=0)            # F(3^3, 2^3): stand-alone pool only
    d2 = wino.Plan(2, 4, 3, 4, 16, [1, 8, 8], pad=1)                # 2-D
    tiny = wino.Plan(3, 4, 3, 4, 16, [1, 1, 8, 8], pad=1)           # Y_0 = 1
    assert fused.desc["fused"] == 1 and two.desc["fused"] == 0
    ws = 1 << 30
    args = (vp(4096), vp(8192), None)
    for w in [(2, 1, 1), (1, 1, 2), (1, 3, 3), (2, 2, 1), (1, 1, 1)]:
        assert L.wino_forward_pool(fused.handle, *args, W(*w), vp(16384), None, 0, None) == -2, w
    assert L.wino_forward_pool(fused.handle, *args, W(0, 2, 2), vp(16384), None, 0, None) == -1
    assert L.wino_forward_pool(fused.handle, *args, None, vp(16384), None, 0, None) == -1
    assert L.wino_forward_pool(fused.handle, vp(4096 + 4), vp(8192), None, W(1, 2, 2), vp(16384), None, 0,
                               None) == -1
    assert L.wino_forward_pool(fused.handle, *args, W(1, 2, 2), vp(16384 + 8), None, 0, None) == -1
    assert L.wino_forward_pool(fused.handle, vp(4096), vp(8192), vp(512 + 2), W(1, 2, 2), vp(16384), None, 0,
                               None) == -1
    assert L.wino_forward_pool(m2.handle, *args, W(1, 2, 2), vp(16384), vp(32768), ws, None) == -2
    assert L.wino_forward_pool(m32.handle, *args, W(2, 2, 2), vp(16384), vp(32768), ws, None) == -2
    assert L.wino_forward_pool(d2.handle, *args, W(1, 2, 2), vp(16384), vp(32768), ws, None) == -2
    assert L.wino_forward_pool(tiny.handle, *args, W(2, 2, 2), vp(16384), None, 0, None) == -1
    # the two-stage product needs its workspace (V)
    assert L.wino_forward_pool(two.handle, *args, W(2, 2, 2), vp(16384), None, 0, None) == -1
    assert L.wino_forward_pool(two.handle, *args, W(2, 2, 2), vp(16384), vp(32768),
                               two.forward_workspace_bytes - 4, None) == -3
    assert fused.pooled_shape((2, 2, 2)) == (1, 16, 4, 4, 4)
    assert fused.pooled_shape((1, 2, 2)) == (1, 16, 8, 4, 4)


def _kappa_from_oracle(N, m, r, pts):
    """kappa of include/wino.h from the oracle's exact matrices (Fractions)."""
    AT, BT, G = winograd_matrices(m, r, pts)
    a = m + r - 1
    gn = [sum(abs(v) for v in G[x]) for x in range(a)]
    bn = [sum(abs(v) for v in BT[x]) for x in range(a)]
    k1 = max(sum(abs(AT[i][x]) * gn[x] * bn[x] for x in range(a)) for i in range(m)) / r
    return float(k1) ** N


@pytest.mark.parametrize("N,m,r,pts", [
    (3, 2, 3, None), (3, 4, 3, None), (3, 4, 3, PAPER_F43_POINTS), (2, 5, 4, None),
    (2, 4, 3, (0, 2, -2, 0.5, -0.5)), (2, 3, 6, (0, 1, -1, 3, -3, Fraction(1, 3), Fraction(-1, 3))),
])
def test_points_error_growth_matches_oracle_matrices(N, m, r, pts):
    got = wino.points_error_growth(N, m, r, pts)
    want = _kappa_from_oracle(N, m, r, pts if pts is not None else default_points(m, r))
    assert abs(got - want) <= 1e-9 * want


@pytest.mark.parametrize("N,m,r", [(3, 2, 3), (3, 4, 3), (2, 4, 3), (2, 5, 4), (2, 4, 5), (2, 3, 6), (2, 3, 2)])
def test_search_points(N, m, r):
    pts, g = wino.search_points(N, m, r)
    assert len(pts) == m + r - 2 and len(set(pts)) == len(pts)
    assert sorted(pts) == sorted(-p for p in pts)                 # symmetric
    assert abs(g - _kappa_from_oracle(N, m, r, [Fraction(p).limit_denominator(64) for p in pts])) <= 1e-9 * g
    assert g <= wino.points_error_growth(N, m, r) * (1 + 1e-12)  # no worse than the default set
    if (m, r) == (4, 3):
        assert g < wino.points_error_growth(N, m, r, PAPER_F43_POINTS)


def test_points_error_growth_rejects(L):
    g = ctypes.c_double()
    two = (ctypes.c_double * 2)(0.0, 1.0)
    assert L.wino_points_error_growth(3, 4, 3, two, 2, ctypes.byref(g)) == -1   # wrong count
    same = (ctypes.c_double * 5)(0.0, 1.0, 1.0, 2.0, -2.0)
    assert L.wino_points_error_growth(3, 4, 3, same, 5, ctypes.byref(g)) == -1  # coincident
    assert L.wino_points_error_growth(0, 4, 3, None, 0, ctypes.byref(g)) == -1
    assert L.wino_points_error_growth(2, 6, 4, None, 0, ctypes.byref(g)) == -1  # alpha 9
    out = (ctypes.c_double * 5)()
    assert L.wino_search_points(3, 4, 3, out, None) == -1


def test_adjoint_plan():
    # the data gradient's plan: C and K swapped, extents Y -> X, pads r - 1 - pad,
    # the forward plan's points and WINO_NO_SPLIT, no ReLU
    f = wino.Plan(3, 2, 3, 16, 24, [2, 9, 10, 11], pad=[1, 0, 2], points=[0, 0.5, -0.5], relu=True,
                  split=False)
    a = f.adjoint()
    assert (a.C, a.K, a.N, a.m, a.r) == (24, 16, 3, 2, 3)
    assert a.input_shape == f.output_shape and a.output_shape == f.input_shape
    assert a.weight_shape == (16, 24, 3, 3, 3)
    assert a.desc["gemm_parts"] == 1
    for u, v in zip(f.matrices(), a.matrices()):
        assert np.array_equal(u, v)
    assert not a.relu
    q = wino.Plan(2, 4, 3, 3, 5, [1, 9, 10], pad=0).adjoint()
    assert q.input_shape == (1, 5, 7, 8) and q.output_shape == (1, 3, 9, 10)
    assert q.desc["default_points"] == 1
    L = wino.lib()
    with pytest.raises(wino.WinoError):
        wino.Plan(2, 2, 3, 3, 5, [1, 9, 10], pad=3).adjoint()       # pad > r - 1
    h = ctypes.c_void_p()
    assert L.wino_plan_adjoint(None, ctypes.byref(h)) == -1
    assert L.wino_plan_adjoint(f.handle, None) == -1
    assert L.wino_transform_filter_adjoint(None, None, None, None) == -1


def test_weight_gradient_host_side():
    # every size: V, then D, then the tile-range partials
    p = wino.Plan(3, 2, 3, 64, 128, [8, 16, 56, 56], pad=1)
    d = p.desc
    v = 4 * 64 * d["C_pad"] * d["T_pad"]
    dbytes = 4 * 64 * 128 * d["T_pad"]
    assert p.weight_gradient_workspace_bytes > v + dbytes
    assert wino.Plan(2, 4, 3, 3, 5, [2, 9, 10], pad=1).weight_gradient_workspace_bytes > 0
    assert wino.Plan(2, 2, 3, 3, 5, [2, 9, 10], pad=4).weight_gradient_workspace_bytes > 0
    for args in [(3, 4, 3), (2, 5, 4), (2, 3, 2), (2, 4, 5), (2, 3, 6), (3, 3, 2)]:
        q = wino.Plan(*args, 3, 5, [1] + [12] * args[0], pad=1)
        assert q.weight_gradient_workspace_bytes > 0, args
    # the 3-D alpha = 8 sizes have no weight gradient
    for args in [(3, 5, 4), (3, 4, 5), (3, 3, 6)]:
        q = wino.Plan(*args, 3, 5, [1] + [12] * args[0], pad=1)
        assert q.weight_gradient_workspace_bytes == 0, args
        assert q.desc["n_xi"] == 512 and q.desc["block_tiles"] == 16 and q.desc["channel_group"] == 4
    L = wino.lib()
    assert L.wino_weight_gradient_workspace_bytes(None) == 0
    assert L.wino_weight_gradient(None, None, None, None, None, 0, None) == -1
    assert L.wino_weight_gradient(p.handle, None, None, None, None, 0, None) == -1


def test_plan_rejects_overflowing_sizes(L):
    """Sizes whose padded counts, byte counts or grids overflow are refused
    before any number is narrowed (the planner computes them in 64 bits)."""
    big = 2 ** 31 - 1
    d = [1, 8, 8, 8]
    assert _plan_status(L, 3, 2, 3, big, 16, d, pad=[1, 1, 1]) == -1
    assert _plan_status(L, 3, 2, 3, 16, big, d, pad=[1, 1, 1]) == -1
    assert _plan_status(L, 3, 4, 3, 16, big - 39, d, pad=[1, 1, 1]) == -1
    assert _plan_status(L, 2, 4, 3, 2 ** 20 + 1, 4, [1, 8, 8]) == -1
    assert _plan_status(L, 2, 4, 3, 2 ** 20, 4, [1, 8, 8]) == 0
    # the two-stage F(4^3) product addresses a wave's U operands from one base:
    # 18 planes of C_pad x K_pad floats stay below 2^32 bytes
    assert _plan_status(L, 3, 4, 3, 7680, 7680, [1, 4, 4, 4], pad=[1, 1, 1]) == 0
    assert _plan_status(L, 3, 4, 3, 7744, 7744, [1, 4, 4, 4], pad=[1, 1, 1]) == -1
    assert _plan_status(L, 3, 2, 3, 4, 4, [big] * 4) == -1
    assert _plan_status(L, 3, 2, 3, 4, 4, [big, 1, 1, 4], pad=[1, 1, 1]) == -1
    assert _plan_status(L, 3, 2, 3, 4, 4, [1, 4, 4, 4], pad=[2 ** 20] * 3) == -1
    vp = ctypes.c_void_p
    win = (ctypes.c_int32 * 3)(2, 2, 2)
    for dims in [(1 << 62, 2, 2, 2), (1 << 40, big, big, big), (1 << 34, 2, 2, 2), (-1, 2, 2, 2)]:
        arr = (ctypes.c_int64 * 4)(*dims)
        assert L.wino_maxpool3d(arr, win, vp(4096), vp(8192), None) == -1, dims


def test_per_axis_tiles_host_side(L):
    """wino_opts.tile: mixed tiles (2, 4, 4) and (4, 2, 2) in 3-D plan; other
    mixes are unsupported, caller points and entries past N are refused."""
    def st(N, m, tile, points=None, dims=None):
        opts = wino._Opts()
        for i, t in enumerate(tile):
            opts.tile[i] = t
        keep = None
        if points is not None:
            keep = (ctypes.c_double * len(points))(*points)
            opts.points = ctypes.cast(keep, ctypes.POINTER(ctypes.c_double))
            opts.n_points = len(points)
        dims = dims or [1] + [9] * N
        arr = (ctypes.c_int64 * len(dims))(*dims)
        h = ctypes.c_void_p()
        s = L.wino_plan(N, m, 3, 4, 4, arr, ctypes.byref(opts), ctypes.byref(h))
        if s == 0:
            L.wino_destroy(h)
        return s
    assert st(3, 4, (2, 0, 0)) == 0
    assert st(3, 2, (4, 2, 2)) == 0
    assert st(3, 2, (0, 4, 4)) == 0          # (2, 4, 4) from m = 2
    assert st(3, 4, (4, 4, 4)) == 0          # isotropic
    assert st(3, 2, (4, 4, 4)) == 0          # isotropic, m = 4 from the tiles
    assert wino.Plan(3, 2, 3, 4, 4, [1, 9, 9, 9], tile=(4, 4, 4)).desc["m"] == 4
    assert st(3, 4, (2, 4, 2)) == -2
    assert st(3, 4, (2, 2, 4)) == -2
    assert st(2, 4, (2, 4, 0)) == -2
    assert st(3, 4, (2, 0, 0), points=(0, 1, -1, 2, -2)) == -1
    assert st(2, 4, (0, 0, 2)) == -1         # entry past N
    assert st(3, 4, (-1, 0, 0)) == -1
    p = wino.Plan(3, 4, 3, 20, 24, [2, 7, 13, 11], pad=1, tile=(2, 4, 4))
    d = p.desc
    assert d["tile"] == [2, 4, 4] and d["alpha_axis"] == [4, 6, 6] and d["alpha"] == 0
    assert d["n_xi"] == 144 and d["tiles"] == [4, 4, 3] and d["T"] == 2 * 4 * 4 * 3
    assert d["fused"] == 0 and p.forward_workspace_bytes == p.workspace_bytes > 0
    assert p.filter_bytes == 4 * 144 * d["C_pad"] * d["K_pad"]
    assert p.weight_gradient_workspace_bytes == 0
    a = p.adjoint()
    assert a.desc["tile"] == [2, 4, 4] and a.input_shape == p.output_shape
    AT = np.zeros(64)
    P = ctypes.POINTER(ctypes.c_double)
    assert L.wino_get_matrices(p.handle, AT.ctypes.data_as(P), None, None) == -2
    q = wino.Plan(3, 2, 3, 3, 5, [1, 9, 6, 7], tile=(4, 2, 2))
    assert q.desc["tile"] == [4, 2, 2] and q.desc["n_xi"] == 96 and q.output_shape == (1, 5, 7, 4, 5)
