"""GPU tests of wino_forward_pool: the F(4^3) forward, fused or in two
stages, with the C3D stack's max-pool (windows (1, 2, 2) and (2, 2, 2),
window = stride, floor rounding) in the product's epilogue, and the F(2^3)
forward with window (2, 2, 2) (one tile per window; the split products'
partial sums reduced and pooled together).

The pooled output must have the same bits as the forward followed by the
stand-alone max-pool (both scan each window in the same order), and match
pool(f(conv + bias)) of the fp64 oracle: the maximum is 1-Lipschitz, so an
output's error is at most the largest error over its window, and the bar is
the m = 4 tolerance against the largest denominator of the window."""
import numpy as np
import pytest

from gpu_util import log, require_gpu
from oracle.direct import direct_blas
from oracle.metric import normalised_error
from oracle.pool import maxpool
from workloads import LayerSpec, draw_layer

pytestmark = pytest.mark.gpu

CASES = [
    # kernel-block loop (C <= 8), rows of whole 16-tile blocks, C3D conv1's window
    (LayerSpec("pool_kloop_row_c3_k64", N=3, m=4, r=3, batch=2, C=3, K=64, X=(8, 12, 64), pad=1,
               x_dist="uniform", w_dist="he", relu=True), (1, 2, 2)),
    # kernel-block loop, gathered rows, odd extents (floor rounding drops the last row)
    (LayerSpec("pool_kloop_c8_k40", N=3, m=4, r=3, batch=1, C=8, K=40, X=(10, 9, 13), pad=1,
               x_dist="normal", w_dist="he", relu=True), (2, 2, 2)),
    # kernel-block loop with at most 4 channels (one MFMA k-step per element), gathered rows
    (LayerSpec("pool_kloop_narrow_c2_k48", N=3, m=4, r=3, batch=1, C=2, K=48, X=(10, 11, 13), pad=1,
               x_dist="normal", w_dist="he", leaky=0.125), (2, 2, 2)),
    # chunk loop (C > 8), partial tiles on every axis, leaky activation
    (LayerSpec("pool_c17_k20_leaky", N=3, m=4, r=3, batch=1, C=17, K=20, X=(9, 10, 11), pad=1,
               x_dist="normal", w_dist="he", leaky=0.125), (2, 2, 2)),
    (LayerSpec("pool_c33_k48_pad0", N=3, m=4, r=3, batch=2, C=33, K=48, X=(7, 13, 10), pad=0,
               x_dist="relu_normal", w_dist="he", relu=True), (1, 2, 2)),
    # no activation: negative maxima survive
    (LayerSpec("pool_c12_k16_noact", N=3, m=4, r=3, batch=1, C=12, K=16, X=(6, 8, 64), pad=2,
               x_dist="normal", w_dist="normal"), (2, 2, 2)),
]
# the two-stage product (k_gemm_inv): K > 64, or the fused form switched off
TWO_STAGE = [
    (LayerSpec("pool2s_c24_k80", N=3, m=4, r=3, batch=1, C=24, K=80, X=(8, 11, 9), pad=1,
               x_dist="relu_normal", w_dist="he", relu=True), (1, 2, 2)),
    (LayerSpec("pool2s_c64_k128", N=3, m=4, r=3, batch=2, C=64, K=128, X=(8, 12, 16), pad=1,
               x_dist="relu_normal", w_dist="he", relu=True), (2, 2, 2)),
    (LayerSpec("pool2s_c17_k20_leaky", N=3, m=4, r=3, batch=1, C=17, K=20, X=(9, 10, 11), pad=1,
               x_dist="normal", w_dist="he", leaky=0.125), (2, 2, 2)),
    (LayerSpec("pool2s_c5_k16_noact", N=3, m=4, r=3, batch=1, C=5, K=16, X=(7, 9, 13), pad=0,
               x_dist="normal", w_dist="normal"), (1, 2, 2)),
]
# F(2^3), window (2, 2, 2): split products (every block of these small layers
# is a tail block, reduced by k_part_reduce_pool) and unsplit ones (the
# pooled epilogue of k_gemm_acc); odd extents drop the last tile row
M2 = [
    (LayerSpec("pool_m2_c16_k64", N=3, m=2, r=3, batch=2, C=16, K=64, X=(8, 12, 16), pad=1,
               x_dist="relu_normal", w_dist="he", relu=True), True),
    (LayerSpec("pool_m2_c16_k64_unsplit", N=3, m=2, r=3, batch=2, C=16, K=64, X=(8, 12, 16), pad=1,
               x_dist="relu_normal", w_dist="he", relu=True), False),
    (LayerSpec("pool_m2_c24_k80_odd", N=3, m=2, r=3, batch=1, C=24, K=80, X=(7, 9, 13), pad=1,
               x_dist="normal", w_dist="he", leaky=0.125), True),
    (LayerSpec("pool_m2_c24_k80_odd_unsplit", N=3, m=2, r=3, batch=1, C=24, K=80, X=(7, 9, 13), pad=1,
               x_dist="normal", w_dist="he", leaky=0.125), False),
    (LayerSpec("pool_m2_c5_k16_pad0_noact", N=3, m=2, r=3, batch=1, C=5, K=16, X=(9, 10, 11), pad=0,
               x_dist="normal", w_dist="normal"), True),
]


def _run(spec, window, seed, bias=True, fuse=True, split=True):
    torch = require_gpu()
    from paper_1611_06565_amd.wino import Plan, maxpool3d
    log(f"[gpu] {spec.name} window={window} C={spec.C} K={spec.K} X={spec.X} pad={spec.pad}")
    x, w = draw_layer(spec, seed=seed)
    b = (0.25 * np.random.default_rng(seed + 1).standard_normal(spec.K)).astype(np.float32) if bias else None
    plan = Plan(spec.N, spec.m, spec.r, spec.C, spec.K, [spec.batch] + list(spec.X), pad=spec.pad,
                relu=spec.relu, leaky=spec.leaky, fuse=fuse, split=split)
    assert plan.desc["fused"] == (1 if fuse and spec.m == 4 and spec.K <= 64 else 0)
    if spec.m == 2:
        assert (plan.desc["gemm_parts"] > 1) == split, plan.desc
    xd = torch.from_numpy(x).cuda()
    U = plan.transform_filter(torch.from_numpy(w).cuda())
    bd = torch.from_numpy(b).cuda() if bias else None
    shape = plan.pooled_shape(window)
    n = int(np.prod(shape))
    guard = 256
    buf = torch.full((n + 2 * guard,), 12345.5, dtype=torch.float32, device="cuda")
    yp = buf[guard:guard + n].view(shape)
    plan.forward_pool(xd, U, window, y=yp, bias=bd)
    y2 = maxpool3d(plan.forward(xd, U, bias=bd), window)
    torch.cuda.synchronize()
    hb = buf.cpu().numpy()
    assert np.all(hb[:guard] == 12345.5) and np.all(hb[-guard:] == 12345.5), "guard band written"
    return x, w, b, yp.cpu().numpy(), y2.cpu().numpy()


@pytest.mark.parametrize("spec,window,fuse,split",
                         [c + (True, True) for c in CASES] + [c + (False, True) for c in TWO_STAGE]
                         + [(c[0], (2, 2, 2), False, c[1]) for c in M2],
                         ids=[c[0].name for c in CASES] + [c[0].name for c in TWO_STAGE] + [c[0].name for c in M2])
def test_forward_pool_matches_forward_then_pool_and_oracle(spec, window, fuse, split):
    x, w, b, yp, y2 = _run(spec, window, seed=41, fuse=fuse, split=split)
    assert yp.shape == y2.shape
    assert np.array_equal(yp.view(np.uint32), y2.view(np.uint32)), "fused pool differs from forward + pool"
    y_ref, den = direct_blas(x, w, spec.pad, relu=spec.relu, bias=b, leaky=spec.leaky)
    ref_p = maxpool(y_ref, window)
    den_p = maxpool(den, window)          # the window's largest denominator
    err = normalised_error(yp, ref_p, den_p)
    log(f"  pooled max err {err['max']:.3e} at {err['argmax']}")
    assert err["nonfinite"] == 0 and err["max"] <= (1e-5 if spec.m == 2 else 1e-4), err


def test_forward_pool_determinism_bitwise():
    spec, window = CASES[2]
    _, _, _, a, _ = _run(spec, window, seed=42)
    _, _, _, c, _ = _run(spec, window, seed=42)
    assert np.array_equal(a.view(np.uint32), c.view(np.uint32))


def test_forward_pool_refusals():
    torch = require_gpu()
    from paper_1611_06565_amd.wino import Plan, WinoError
    spec = CASES[0][0]
    x, w = draw_layer(spec, seed=43)
    xd = torch.from_numpy(x).cuda()
    # a window the epilogue does not take, and an invalid one
    p1 = Plan(3, 4, 3, spec.C, spec.K, [spec.batch] + list(spec.X), pad=1, relu=True)
    U1 = p1.transform_filter(torch.from_numpy(w).cuda())
    with pytest.raises(WinoError):
        p1.forward_pool(xd, U1, (2, 1, 1))
    with pytest.raises(WinoError):
        p1.forward_pool(xd, U1, (1, 3, 3))
    # F(2^3) takes window (2, 2, 2) only
    p3 = Plan(3, 2, 3, spec.C, spec.K, [spec.batch] + list(spec.X), pad=1, relu=True)
    U3 = p3.transform_filter(torch.from_numpy(w).cuda())
    with pytest.raises(WinoError):
        p3.forward_pool(xd, U3, (1, 2, 2))
    torch.cuda.synchronize()


def test_forward_pool_full_size_conv1_bitwise():
    """conv1 of the C3D stack at full size (batch 4, C = 3, K = 64,
    16 x 112 x 112, window (1, 2, 2)): the fused pool has the bits of the
    forward followed by the stand-alone pool on every output."""
    torch = require_gpu()
    from paper_1611_06565_amd.wino import Plan, maxpool3d
    from workloads import C3D_STACK, draw_stack
    (spec, pool), = [lp for lp in C3D_STACK.layers()][:1]
    x, ws = draw_stack(C3D_STACK, seed=5)
    log(f"[gpu] full-size conv1 C={spec.C} K={spec.K} X={spec.X} window={pool.window}")
    plan = Plan(3, 4, 3, spec.C, spec.K, [spec.batch] + list(spec.X), pad=1, relu=True)
    assert plan.desc["fused"] == 1
    xd = torch.from_numpy(x).cuda()
    U = plan.transform_filter(torch.from_numpy(ws[0]).cuda())
    yp = plan.forward_pool(xd, U, pool.window)
    y2 = maxpool3d(plan.forward(xd, U), pool.window)
    torch.cuda.synchronize()
    assert torch.equal(yp.view(torch.int32), y2.view(torch.int32))


def test_forward_pool_full_size_conv2_two_stage_bitwise():
    """conv2 of the C3D stack at full size (batch 4, C = 64, K = 128,
    16 x 56 x 56, window (2, 2, 2), two-stage F(4^3)): the pooled product has
    the bits of the forward followed by the stand-alone pool."""
    torch = require_gpu()
    from paper_1611_06565_amd.wino import Plan, maxpool3d
    from workloads import C3D_STACK
    spec, pool = list(C3D_STACK.layers())[1]
    log(f"[gpu] full-size conv2 C={spec.C} K={spec.K} X={spec.X} window={pool.window}")
    rng = np.random.default_rng(6)
    x = np.maximum(rng.standard_normal((spec.batch, spec.C) + tuple(spec.X)), 0).astype(np.float32)
    w = (rng.standard_normal((spec.K, spec.C, 3, 3, 3)) * np.sqrt(2.0 / (27 * spec.C))).astype(np.float32)
    plan = Plan(3, 4, 3, spec.C, spec.K, [spec.batch] + list(spec.X), pad=1, relu=True)
    assert plan.desc["fused"] == 0
    xd = torch.from_numpy(x).cuda()
    U = plan.transform_filter(torch.from_numpy(w).cuda())
    yp = plan.forward_pool(xd, U, pool.window)
    y2 = maxpool3d(plan.forward(xd, U), pool.window)
    torch.cuda.synchronize()
    assert torch.equal(yp.view(torch.int32), y2.view(torch.int32))


@pytest.mark.parametrize("name,C,K,X,batch", [
    ("config2_layer", 64, 128, (16, 56, 56), 8),      # whole blocks and split tail blocks
    ("c3d_conv6_shape", 512, 512, (4, 14, 14), 4),    # every block split
    ("c3d_conv8_shape", 512, 512, (2, 7, 7), 4),      # split, odd extents (floor)
])
def test_forward_pool_m2_full_size_bitwise(name, C, K, X, batch):
    """F(2^3) with window (2, 2, 2) at full size: the pooled product has the
    bits of the forward followed by the stand-alone pool on every output."""
    torch = require_gpu()
    from paper_1611_06565_amd.wino import Plan, maxpool3d
    log(f"[gpu] full-size F(2^3) pooled {name} C={C} K={K} X={X} batch={batch}")
    rng = np.random.default_rng(7)
    x = np.maximum(rng.standard_normal((batch, C) + tuple(X)), 0).astype(np.float32)
    w = (rng.standard_normal((K, C, 3, 3, 3)) * np.sqrt(2.0 / (27 * C))).astype(np.float32)
    b = (0.1 * rng.standard_normal(K)).astype(np.float32)
    plan = Plan(3, 2, 3, C, K, [batch] + list(X), pad=1, relu=True)
    xd = torch.from_numpy(x).cuda()
    bd = torch.from_numpy(b).cuda()
    U = plan.transform_filter(torch.from_numpy(w).cuda())
    yp = plan.forward_pool(xd, U, (2, 2, 2), bias=bd)
    y2 = maxpool3d(plan.forward(xd, U, bias=bd), (2, 2, 2))
    torch.cuda.synchronize()
    assert torch.equal(yp.view(torch.int32), y2.view(torch.int32))
