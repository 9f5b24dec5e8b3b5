"""GPU parity of 3-D layers with per-axis output tiles (eq. 4 with its own
transform triple per axis): F(2,3) on the first axis and F(4,3) on the other
two, and the reverse, through the C ABI against the fp64 direct correlation
on every output.  Bar: the m = 4 bar (1e-4 normalised), since F(4,3) runs on
at least one axis.  Also: the transformed kernels and inputs against the
oracle's per-axis steps, the data gradient through the adjoint plan, and
bitwise run-to-run determinism."""
import numpy as np
import pytest

from gpu_util import check_full, log, require_gpu, run_layer, tol
from oracle.adjoint import direct_adjoint
from oracle.metric import normalised_error
from oracle.winograd import transform_filter as o_filter
from oracle.winograd import transform_input as o_input
from workloads import LayerSpec, draw_layer

pytestmark = pytest.mark.gpu

SMALL = [
    LayerSpec("ax244_ragged", N=3, m=4, r=3, batch=2, C=20, K=24, X=(7, 13, 11), pad=1,
              x_dist="normal", w_dist="he", tile=(2, 4, 4)),
    LayerSpec("ax422_ragged", N=3, m=2, r=3, batch=1, C=18, K=40, X=(11, 9, 10), pad=1,
              x_dist="uniform", w_dist="he", tile=(4, 2, 2)),
    LayerSpec("ax244_pad0_relu", N=3, m=4, r=3, batch=1, C=5, K=7, X=(4, 9, 8), pad=0,
              x_dist="normal", w_dist="normal", relu=True, tile=(2, 4, 4)),
    LayerSpec("ax422_pad2_leaky", N=3, m=2, r=3, batch=2, C=33, K=17, X=(5, 6, 7), pad=2,
              x_dist="normal", w_dist="he", leaky=0.1, tile=(4, 2, 2)),
    LayerSpec("ax244_one_tile", N=3, m=4, r=3, batch=1, C=3, K=2, X=(3, 5, 4), pad=0,
              x_dist="normal", w_dist="normal", tile=(2, 4, 4)),
    LayerSpec("ax244_k48_c40", N=3, m=4, r=3, batch=3, C=40, K=48, X=(6, 10, 12), pad=1,
              x_dist="relu_normal", w_dist="he", tile=(2, 4, 4)),
]

# two C3D-style layers with short temporal extents (conv3/conv4 and conv5/conv6
# shapes of the eight-layer stack at batch 4): 2 on time, 4 on space
C3D_LIKE = [
    LayerSpec("ax244_c3d_conv4", N=3, m=4, r=3, batch=4, C=256, K=256, X=(8, 28, 28), pad=1,
              x_dist="uniform", w_dist="he", relu=True, tile=(2, 4, 4)),
    LayerSpec("ax244_c3d_conv6", N=3, m=4, r=3, batch=4, C=512, K=512, X=(4, 14, 14), pad=1,
              x_dist="uniform", w_dist="he", relu=True, tile=(2, 4, 4)),
]


@pytest.mark.parametrize("spec", SMALL, ids=lambda s: s.name)
def test_aniso_small_full_output(spec):
    x, w = draw_layer(spec, seed=31)
    b = (0.3 * np.random.default_rng(2).standard_normal(spec.K)).astype(np.float32)
    y, plan = run_layer(spec, x, w, guard=512, bias=b)
    d = plan.desc
    assert d["tile"] == list(spec.tile) and d["alpha"] == 0
    assert d["n_xi"] == int(np.prod([t + 2 for t in spec.tile]))
    assert y.shape == (spec.batch, spec.K) + spec.out_spatial
    check_full(spec, y, x, w, bias=b)


@pytest.mark.parametrize("spec", C3D_LIKE, ids=lambda s: s.name)
def test_aniso_c3d_layers_full_output(spec):
    x, w = draw_layer(spec, seed=37)
    y, _ = run_layer(spec, x, w)
    assert np.all(np.isfinite(y))
    check_full(spec, y, x, w)


@pytest.mark.parametrize("spec", SMALL[:2], ids=lambda s: s.name)
def test_aniso_transform_stages_match_oracle(spec):
    """U and V on their own against the oracle's per-axis steps 2 and 3."""
    torch = require_gpu()
    from paper_1611_06565_amd.wino import Plan
    x, w = draw_layer(spec, seed=8)
    plan = Plan(spec.N, spec.m, spec.r, spec.C, spec.K, [spec.batch] + list(spec.X), pad=spec.pad,
                tile=spec.tile)
    d = plan.desc
    U = plan.transform_filter(torch.from_numpy(w).cuda())
    ws = plan.transform_input(torch.from_numpy(x).cuda())
    torch.cuda.synchronize()
    nxi = d["n_xi"]
    Ug = plan.unpack_filter(U)
    Vg = plan.unpack_workspace(ws)
    Uo = o_filter(w, spec.tile, spec.r).reshape(spec.K, spec.C, nxi).transpose(2, 1, 0)
    Vo = o_input(x, spec.tile, spec.r, spec.pad).reshape(d["T"], spec.C, nxi).transpose(2, 1, 0)
    assert np.all(Ug[:, spec.C:, :] == 0) and np.all(Ug[:, :, spec.K:] == 0)
    assert np.all(Vg[:, spec.C:, :] == 0) and np.all(Vg[:, :, d["T"]:] == 0)
    assert np.abs(Ug[:, :spec.C, :spec.K] - Uo).max() <= 1e-6 * (np.abs(Uo).max() + 1e-30)
    assert np.abs(Vg[:, :spec.C, :d["T"]] - Vo).max() <= 1e-6 * (np.abs(Vo).max() + 1e-30)


@pytest.mark.parametrize("spec", SMALL[:2], ids=lambda s: s.name)
def test_aniso_data_gradient(spec):
    """dx through the adjoint plan (same per-axis tiles, flipped kernels)."""
    torch = require_gpu()
    from paper_1611_06565_amd.wino import Plan
    rng = np.random.default_rng(9)
    plan = Plan(spec.N, spec.m, spec.r, spec.C, spec.K, [spec.batch] + list(spec.X), pad=spec.pad,
                tile=spec.tile)
    adj = plan.adjoint()
    assert adj.desc["tile"] == list(spec.tile)
    w = (0.2 * rng.standard_normal(plan.weight_shape)).astype(np.float32)
    dy = rng.standard_normal(plan.output_shape).astype(np.float32)
    U = adj.transform_filter_adjoint(torch.from_numpy(w).cuda())
    dx = adj.forward(torch.from_numpy(dy).cuda(), U)
    torch.cuda.synchronize()
    ref, den = direct_adjoint(dy, w, spec.pad)
    err = normalised_error(dx.cpu().numpy(), ref, den)
    log(f"  adjoint max err {err['max']:.3e}")
    assert err["nonfinite"] == 0 and err["max"] <= tol(spec), err


def test_aniso_determinism_bitwise():
    spec = SMALL[0]
    x, w = draw_layer(spec, seed=2)
    y1, _ = run_layer(spec, x, w)
    y2, _ = run_layer(spec, x, w)
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))
