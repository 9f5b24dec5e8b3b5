"""The library's calls under HIP graph capture: every forward launches kernels
only (no allocation, no memset), so a captured forward, data gradient or
weight gradient replays to the bits of the eager call.  Each graph is replayed
several times with eager work and synchronisations between the replays, and
every replay is checked."""
import numpy as np
import pytest

from gpu_util import log, require_gpu
from workloads import LayerSpec, draw_layer

pytestmark = pytest.mark.gpu

CASES = [
    # F(2^3) with the tail split (partial outputs + k_part_reduce), and without
    (LayerSpec("g_f2x3_parts", N=3, m=2, r=3, batch=2, C=96, K=130, X=(4, 10, 9), pad=1,
               x_dist="normal", w_dist="he"), {"split": True}),
    (LayerSpec("g_f2x3_nosplit", N=3, m=2, r=3, batch=2, C=24, K=40, X=(6, 13, 15), pad=1,
               x_dist="normal", w_dist="he", relu=True), {"split": False}),
    # F(4^2): tail blocks split into parts of 1 or 2 of its 18 passes
    (LayerSpec("g_f4x3_2d", N=2, m=4, r=3, batch=3, C=36, K=70, X=(17, 23), pad=1,
               x_dist="normal", w_dist="he"), {"split": True}),
    # F(4^3): k_fused43, and k_input_split + k_gemm_inv
    (LayerSpec("g_f4x3_3d_fused", N=3, m=4, r=3, batch=1, C=20, K=24, X=(13, 11, 17), pad=1,
               x_dist="normal", w_dist="he"), {"split": True, "fuse": True}),
    (LayerSpec("g_f4x3_3d_two_stage", N=3, m=4, r=3, batch=1, C=20, K=24, X=(13, 11, 17), pad=1,
               x_dist="normal", w_dist="he"), {"split": True, "fuse": False}),
    # per-axis tiles F(2,3) x F(4,3)^2
    (LayerSpec("g_aniso_244", N=3, m=2, r=3, batch=2, C=12, K=20, X=(10, 15, 13), pad=1,
               x_dist="normal", w_dist="he", tile=(2, 4, 4)), {"split": True}),
]


def _replay_check(torch, graph, out, eager, scratch):
    for rep in range(4):
        scratch.mul_(1.0001)                        # eager work between replays
        torch.cuda.synchronize()
        out.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {rep} differs"


@pytest.mark.parametrize("spec,kw", CASES, ids=[c[0].name for c in CASES])
def test_forward_graph_replay(spec, kw):
    torch = require_gpu()
    from paper_1611_06565_amd.wino import Plan
    log(f"[gpu] graph forward {spec.name} {kw}")
    x, w = draw_layer(spec, seed=21)
    plan = Plan(spec.N, spec.m, spec.r, spec.C, spec.K, [spec.batch] + list(spec.X), pad=spec.pad,
                relu=spec.relu, tile=spec.tile, **kw)
    if "fuse" in kw:
        assert plan.desc["fused"] == (1 if kw["fuse"] else 0)
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    U = plan.transform_filter(wd)
    ws = plan.new_workspace()
    y = plan.new_output()
    plan.forward(xd, U, y=y, workspace=ws)
    torch.cuda.synchronize()
    eager = y.clone()
    scratch = torch.ones(1 << 20, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):                      # warm-up on the side stream
        plan.forward(xd, U, y=y, workspace=ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        plan.forward(xd, U, y=y, workspace=ws)
    _replay_check(torch, g, y, eager, scratch)


def test_gradients_graph_replay():
    torch = require_gpu()
    from paper_1611_06565_amd.wino import Plan
    log("[gpu] graph gradients")
    spec = CASES[0][0]
    x, w = draw_layer(spec, seed=22)
    plan = Plan(spec.N, spec.m, spec.r, spec.C, spec.K, [spec.batch] + list(spec.X), pad=spec.pad)
    adj = plan.adjoint()
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    dyd = torch.from_numpy(np.random.default_rng(3).standard_normal(plan.output_shape, dtype=np.float32)).cuda()
    Ua = adj.transform_filter_adjoint(wd)
    wsa = adj.new_workspace()
    dx = adj.new_output()
    wsw = torch.empty(plan.weight_gradient_workspace_bytes // 4, device="cuda")
    dw = torch.empty(plan.weight_shape, device="cuda")
    adj.forward(dyd, Ua, y=dx, workspace=wsa)
    plan.weight_gradient(xd, dyd, dw, wsw)
    torch.cuda.synchronize()
    dx_e, dw_e = dx.clone(), dw.clone()
    scratch = torch.ones(1 << 20, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        adj.forward(dyd, Ua, y=dx, workspace=wsa)
        plan.weight_gradient(xd, dyd, dw, wsw)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    ga, gw = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(ga):
        adj.forward(dyd, Ua, y=dx, workspace=wsa)
    with torch.cuda.graph(gw):
        plan.weight_gradient(xd, dyd, dw, wsw)
    _replay_check(torch, ga, dx, dx_e, scratch)
    _replay_check(torch, gw, dw, dw_e, scratch)


@pytest.mark.parametrize("case,fuse,window,split",
                         [(3, True, (1, 2, 2), True), (3, False, (2, 2, 2), True),
                          (0, False, (2, 2, 2), True), (1, False, (2, 2, 2), False)],
                         ids=["fused_122", "two_stage_222", "f2x3_parts_222", "f2x3_nosplit_222"])
def test_forward_pool_graph_replay(case, fuse, window, split):
    """wino_forward_pool under capture: the fused F(4^3) forward, the
    two-stage one and the F(2^3) one (split into parts reduced and pooled
    together, and unsplit), each with the max-pool in the product."""
    torch = require_gpu()
    from paper_1611_06565_amd.wino import Plan
    spec = CASES[case][0]
    log(f"[gpu] graph forward_pool {spec.name} fuse={fuse} window={window} split={split}")
    x, w = draw_layer(spec, seed=23)
    plan = Plan(spec.N, spec.m, spec.r, spec.C, spec.K, [spec.batch] + list(spec.X), pad=spec.pad,
                relu=True, fuse=fuse, split=split)
    assert plan.desc["fused"] == (1 if fuse else 0)
    if case == 0:
        assert plan.desc["gemm_parts"] > 1, "the split case must split"
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    U = plan.transform_filter(wd)
    ws = plan.new_workspace() if not fuse else None
    y = torch.empty(plan.pooled_shape(window), device="cuda")
    plan.forward_pool(xd, U, window, y=y, workspace=ws)
    torch.cuda.synchronize()
    eager = y.clone()
    scratch = torch.ones(1 << 20, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        plan.forward_pool(xd, U, window, y=y, workspace=ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        plan.forward_pool(xd, U, window, y=y, workspace=ws)
    _replay_check(torch, g, y, eager, scratch)
