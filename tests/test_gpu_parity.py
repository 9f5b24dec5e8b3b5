"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle.

Bar: normalised max error |y - y_ref| / sum|w||x| <= 1e-5 for m = 2 and
<= 1e-4 for m = 4, against the direct correlation of eq. (2).  Every layer,
the full-size workloads in the launch configuration the bench times included,
is compared on every output (the fp64 per-offset BLAS oracle runs the largest
in seconds); the max error, its position and the 99.99th percentile are logged.
Integer inputs with F(2^N, 3^N) must match the integer correlation bit for bit
(every intermediate is a small dyadic rational, exact in fp32).
"""
import numpy as np
import pytest

from gpu_util import check_full, check_sampled, log, require_gpu, run_layer
from oracle.direct import direct_blas
from oracle.pool import maxpool
from oracle.toomcook import PAPER_F43_POINTS
from oracle.winograd import transform_filter as o_filter
from oracle.winograd import transform_input as o_input
from workloads import C3D_STACK, CONFIGS, LayerSpec, draw_layer, draw_stack, fig4_layers

pytestmark = pytest.mark.gpu

SMALL = [
    CONFIGS[1],
    LayerSpec("f2x3_3d_ragged", N=3, m=2, r=3, batch=2, C=24, K=40, X=(6, 13, 15), pad=1,
              x_dist="relu_normal", w_dist="he"),
    LayerSpec("f4x3_2d_ragged", N=2, m=4, r=3, batch=3, C=36, K=70, X=(17, 23), pad=1,
              x_dist="relu_normal", w_dist="he"),
    LayerSpec("f4x3_3d_ragged", N=3, m=4, r=3, batch=1, C=20, K=24, X=(13, 11, 17), pad=1,
              x_dist="uniform", w_dist="he"),
    LayerSpec("f2x3_2d_ragged", N=2, m=2, r=3, batch=2, C=10, K=33, X=(19, 14), pad=1,
              x_dist="normal", w_dist="normal"),
    LayerSpec("f2x3_3d_relu", N=3, m=2, r=3, batch=1, C=16, K=48, X=(9, 10, 11), pad=1,
              x_dist="normal", w_dist="he", relu=True),
    LayerSpec("f4x3_3d_relu", N=3, m=4, r=3, batch=2, C=8, K=16, X=(7, 9, 6), pad=1,
              x_dist="normal", w_dist="he", relu=True),
    # F(4^2) with a fused ReLU: whole blocks only (no split tail), several
    # channel stages and kernel blocks
    LayerSpec("f4x2_2d_relu", N=2, m=4, r=3, batch=3, C=40, K=75, X=(22, 29), pad=1,
              x_dist="normal", w_dist="he", relu=True),
]

# C_pad a multiple of 64: the m = 2 GEMM overlaps each pass's epilogue with
# the next pass (one or two rotations of the four stage buffers per pass)
OVERLAP = [
    LayerSpec("f2x3_3d_c64_ovl", N=3, m=2, r=3, batch=1, C=64, K=70, X=(6, 9, 10), pad=1,
              x_dist="relu_normal", w_dist="he"),
    LayerSpec("f2x3_3d_c128_ovl", N=3, m=2, r=3, batch=2, C=128, K=64, X=(5, 7, 6), pad=1,
              x_dist="normal", w_dist="he", relu=True),
    LayerSpec("f2x3_2d_c64_ovl", N=2, m=2, r=3, batch=3, C=60, K=130, X=(21, 17), pad=1,
              x_dist="uniform", w_dist="he"),
]

EDGE = [
    LayerSpec("one_output", N=3, m=2, r=3, batch=1, C=3, K=2, X=(3, 3, 3), pad=0),
    LayerSpec("one_output_m4", N=3, m=4, r=3, batch=1, C=3, K=2, X=(3, 3, 3), pad=0),
    LayerSpec("c1k1", N=3, m=2, r=3, batch=1, C=1, K=1, X=(5, 7, 4), pad=1),
    LayerSpec("c1k1_2d_m4", N=2, m=4, r=3, batch=1, C=1, K=1, X=(5, 7), pad=1),
    LayerSpec("wide_k", N=3, m=2, r=3, batch=1, C=2, K=130, X=(4, 5, 6), pad=1),
    LayerSpec("pad2", N=3, m=2, r=3, batch=1, C=5, K=7, X=(5, 6, 7), pad=2),
    LayerSpec("pad2_m4_2d", N=2, m=4, r=3, batch=2, C=5, K=7, X=(5, 6), pad=2),
    LayerSpec("batch5", N=3, m=2, r=3, batch=5, C=6, K=9, X=(3, 5, 4), pad=1),
    LayerSpec("tiny_2d", N=2, m=2, r=3, batch=1, C=3, K=3, X=(3, 4), pad=0),
    LayerSpec("odd_c_2d", N=2, m=4, r=3, batch=2, C=7, K=33, X=(12, 9), pad=1),
    LayerSpec("odd_c_3d_m4", N=3, m=4, r=3, batch=1, C=5, K=17, X=(8, 6, 10), pad=1),
]

# F(4^3) with whole rows of 16 tiles along the last axis: the input transform
# loads each block's rows with one aligned 16-byte load per lane and takes the
# window halo from neighbouring lanes (pads 0, 1, 2; one and two blocks per
# row; padding channel groups)
ROWFAST = [
    LayerSpec("f4x3_row1_pad1", N=3, m=4, r=3, batch=2, C=9, K=20, X=(5, 6, 64), pad=1,
              x_dist="normal", w_dist="he"),
    LayerSpec("f4x3_row2_pad1", N=3, m=4, r=3, batch=1, C=4, K=16, X=(3, 4, 128), pad=1,
              x_dist="uniform", w_dist="he", relu=True),
    LayerSpec("f4x3_row1_pad0", N=3, m=4, r=3, batch=1, C=6, K=7, X=(6, 7, 64), pad=0,
              x_dist="normal", w_dist="normal"),
    LayerSpec("f4x3_row1_pad2", N=3, m=4, r=3, batch=1, C=17, K=5, X=(4, 5, 60), pad=2,
              x_dist="normal", w_dist="he"),
]


@pytest.mark.parametrize("spec", SMALL + OVERLAP + EDGE + ROWFAST, ids=lambda s: s.name)
def test_small_layers_full_output(spec):
    x, w = draw_layer(spec, seed=11)
    y, _ = run_layer(spec, x, w, guard=1024)
    assert y.shape == (spec.batch, spec.K) + spec.out_spatial
    check_full(spec, y, x, w)


# F(4^3) forward in both forms: the input transform fused into the product
# (k_fused43, planned for at most 64 kernels) and the two stages through V
# (k_input_split + k_gemm_inv); row-aligned and gathered loads, padding
# channels in the last 8-channel chunk, 1 to 4 kernel blocks, pads 0 to 2
F43_BOTH = [s for s in SMALL + EDGE + ROWFAST if s.N == 3 and s.m == 4] + [
    LayerSpec("f4x3_k64_c40", N=3, m=4, r=3, batch=2, C=40, K=64, X=(9, 10, 12), pad=1,
              x_dist="normal", w_dist="he"),
    LayerSpec("f4x3_k80_two_stage", N=3, m=4, r=3, batch=1, C=24, K=80, X=(8, 11, 9), pad=1,
              x_dist="relu_normal", w_dist="he"),
    LayerSpec("f4x3_row_c33_k48", N=3, m=4, r=3, batch=1, C=33, K=48, X=(6, 5, 64), pad=1,
              x_dist="uniform", w_dist="he"),
    # one chunk of channels (C <= 8) with several kernel blocks: a work-group
    # forms the planes once and runs every kernel block of its tiles
    LayerSpec("f4x3_kloop_row_c3_k64", N=3, m=4, r=3, batch=2, C=3, K=64, X=(6, 7, 64), pad=1,
              x_dist="uniform", w_dist="he"),
    LayerSpec("f4x3_kloop_c8_k40", N=3, m=4, r=3, batch=1, C=8, K=40, X=(9, 10, 11), pad=1,
              x_dist="normal", w_dist="he"),
    LayerSpec("f4x3_kloop_c1_k33", N=3, m=4, r=3, batch=1, C=1, K=33, X=(7, 6, 9), pad=0,
              x_dist="normal", w_dist="normal"),
    # one chunk of 4 and of 5 channels (the chunk's other channels zero)
    LayerSpec("f4x3_kloop_c4_k48", N=3, m=4, r=3, batch=2, C=4, K=48, X=(9, 8, 64), pad=1,
              x_dist="normal", w_dist="he"),
    LayerSpec("f4x3_kloop_c5_k32", N=3, m=4, r=3, batch=1, C=5, K=32, X=(10, 7, 11), pad=2,
              x_dist="normal", w_dist="he"),
    # 300 tile blocks: whole work-groups for every kernel block plus, on each
    # XCD, the blocks past its last full round split into one unit per kernel
    # block
    LayerSpec("f4x3_kloop_tail_c3_k64", N=3, m=4, r=3, batch=1, C=3, K=64, X=(48, 100, 64), pad=1,
              x_dist="relu_normal", w_dist="he"),
]


@pytest.mark.parametrize("spec", F43_BOTH, ids=lambda s: s.name)
def test_f43_fused_and_two_stage(spec):
    x, w = draw_layer(spec, seed=19)
    b = (0.2 * np.random.default_rng(3).standard_normal(spec.K)).astype(np.float32)
    y_f, plan_f = run_layer(spec, x, w, guard=512, bias=b)
    assert plan_f.desc["fused"] == (1 if spec.K <= 64 else 0)
    assert plan_f.forward_workspace_bytes == (0 if spec.K <= 64 else plan_f.workspace_bytes)
    check_full(spec, y_f, x, w, bias=b)
    y_s, plan_s = run_layer(spec, x, w, guard=512, bias=b, fuse=False)
    assert plan_s.desc["fused"] == 0
    check_full(spec, y_s, x, w, bias=b)


def test_f43_fused_determinism_bitwise():
    spec = ROWFAST[0]
    x, w = draw_layer(spec, seed=4)
    y1, p1 = run_layer(spec, x, w)
    y2, _ = run_layer(spec, x, w)
    assert p1.desc["fused"] == 1
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))


def test_f43_fused_integer_inputs():
    """Integer data through the fused F(4^3) kernel: F(4,3)'s matrices hold
    non-dyadic entries, so the bar is the m = 4 tolerance (no bit-exactness),
    but the result must also match the two-stage path within it."""
    spec = LayerSpec("f4x3_int", N=3, m=4, r=3, batch=1, C=16, K=32, X=(8, 9, 64), pad=1,
                     x_dist="int2", w_dist="int2")
    x, w = draw_layer(spec, seed=8)
    y_f, _ = run_layer(spec, x, w)
    y_s, _ = run_layer(spec, x, w, fuse=False)
    check_full(spec, y_f, x, w)
    check_full(spec, y_s, x, w)


# F(5^2, 4^2): alpha = 8, 4 x 4 kernels (the kernel size of the paper's 2-D
# benchmark, §4.4); k_gemm_inv with 64 elements and 25 outputs per (tile, kernel)
F54 = [
    LayerSpec("f5x4_2d_ragged", N=2, m=5, r=4, batch=2, C=9, K=20, X=(23, 31), pad=0,
              x_dist="normal", w_dist="he"),
    LayerSpec("f5x4_2d_pad1_relu", N=2, m=5, r=4, batch=3, C=33, K=17, X=(19, 26), pad=1,
              x_dist="uniform", w_dist="he", relu=True),
    LayerSpec("f5x4_2d_one_tile", N=2, m=5, r=4, batch=1, C=2, K=3, X=(8, 8), pad=0),
    LayerSpec("f5x4_2d_wide", N=2, m=5, r=4, batch=1, C=40, K=70, X=(40, 57), pad=2,
              x_dist="relu_normal", w_dist="he"),
    # the other 2-D sizes of Table 1
    LayerSpec("f4x5_2d", N=2, m=4, r=5, batch=2, C=12, K=19, X=(21, 26), pad=2,
              x_dist="normal", w_dist="he"),
    LayerSpec("f3x6_2d", N=2, m=3, r=6, batch=1, C=20, K=33, X=(25, 19), pad=0,
              x_dist="uniform", w_dist="he", relu=True),
    LayerSpec("f3x2_2d", N=2, m=3, r=2, batch=3, C=17, K=40, X=(20, 23), pad=1,
              x_dist="normal", w_dist="normal"),
]


@pytest.mark.parametrize("spec", F54, ids=lambda s: s.name)
def test_f54_layers_full_output(spec):
    x, w = draw_layer(spec, seed=17)
    y, _ = run_layer(spec, x, w, guard=512)
    assert y.shape == (spec.batch, spec.K) + spec.out_spatial
    check_full(spec, y, x, w)


# F(2^N, 3^N) layers with few product blocks and many channels and kernels
# (the late layers of a 3-D stack): each block's element passes are split over
# up to 32 work-groups whose partial outputs are summed in order afterwards;
# and layers with full rounds of blocks and a few left over (the tail blocks,
# split into 8 parts), with and without ReLU
PARTS = [
    LayerSpec("f2x3_3d_parts_c512", N=3, m=2, r=3, batch=2, C=512, K=192, X=(2, 7, 7), pad=1,
              x_dist="relu_normal", w_dist="he", relu=True),
    LayerSpec("f2x3_3d_parts_ragged", N=3, m=2, r=3, batch=4, C=250, K=150, X=(4, 14, 13), pad=1,
              x_dist="normal", w_dist="he"),
    LayerSpec("f2x3_2d_parts", N=2, m=2, r=3, batch=1, C=300, K=130, X=(15, 14), pad=1,
              x_dist="uniform", w_dist="he"),
    LayerSpec("f2x3_2d_tail_relu", N=2, m=2, r=3, batch=3, C=8, K=64, X=(212, 212), pad=1,
              x_dist="normal", w_dist="he", relu=True),
    LayerSpec("f2x3_3d_tail", N=3, m=2, r=3, batch=1, C=8, K=70, X=(16, 96, 92), pad=1,
              x_dist="relu_normal", w_dist="he"),
    # F(4^2): 18 passes per block, so the parts hold 1 or 2 passes
    LayerSpec("f4x3_2d_parts", N=2, m=4, r=3, batch=2, C=200, K=100, X=(30, 26), pad=1,
              x_dist="normal", w_dist="he", relu=True),
]


@pytest.mark.parametrize("spec", PARTS, ids=lambda s: s.name)
def test_pass_split_layers_full_output(spec):
    x, w = draw_layer(spec, seed=23)
    b = (np.random.default_rng(6).standard_normal(spec.K) * 0.3).astype(np.float32)
    y, plan = run_layer(spec, x, w, bias=b, guard=1024)
    assert plan.desc["gemm_parts"] > 1 and plan.desc["gemm_tail_blocks"] > 0, plan.desc
    check_full(spec, y, x, w, bias=b)
    # the same layer with every block in one work-group
    y1, plan1 = run_layer(spec, x, w, bias=b, guard=1024, split=False)
    assert plan1.desc["gemm_parts"] == 1
    check_full(spec, y1, x, w, bias=b)


def test_pass_split_determinism_bitwise():
    spec = PARTS[1]
    x, w = draw_layer(spec, seed=3)
    b = np.linspace(-1, 1, spec.K).astype(np.float32)
    y1, _ = run_layer(spec, x, w, bias=b)
    y2, _ = run_layer(spec, x, w, bias=b)
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))


# the small F(2^N, 3^N) layers above take the pass split; here every block is
# one work-group again
M2_WHOLE = [s for s in SMALL + OVERLAP + EDGE if s.m == 2]


@pytest.mark.parametrize("spec", M2_WHOLE, ids=lambda s: s.name)
def test_small_m2_layers_no_split(spec):
    x, w = draw_layer(spec, seed=11)
    y, plan = run_layer(spec, x, w, guard=1024, split=False)
    assert plan.desc["gemm_parts"] == 1
    check_full(spec, y, x, w)


# eq. (2)'s bias: every GEMM kernel, with the tail blocks split into parts (the
# bias joins their sum) and with every block whole
BIAS = [SMALL[1], SMALL[5], SMALL[2], SMALL[7], SMALL[3], SMALL[6], F54[0]]


@pytest.mark.parametrize("split", [True, False], ids=["split", "nosplit"])
@pytest.mark.parametrize("spec", BIAS, ids=lambda s: s.name)
def test_bias(spec, split):
    x, w = draw_layer(spec, seed=13)
    b = (np.random.default_rng(4).standard_normal(spec.K) * 0.5).astype(np.float32)
    y, _ = run_layer(spec, x, w, bias=b, guard=256, split=split)
    check_full(spec, y, x, w, bias=b)


# a leaky ReLU as eq. (2)'s activation f (after the bias) on every product
# kernel: k_gemm_acc with and without split tails (k_part_reduce applies it to
# the summed parts), k_gemm_acc4, k_gemm_inv in 3-D and in 2-D (alpha = 8)
LEAKY = [
    LayerSpec("f2x3_3d_leaky", N=3, m=2, r=3, batch=2, C=24, K=70, X=(9, 10, 11), pad=1,
              x_dist="normal", w_dist="he", leaky=0.1),
    LayerSpec("f2x3_2d_leaky_neg", N=2, m=2, r=3, batch=3, C=20, K=33, X=(19, 24), pad=1,
              x_dist="normal", w_dist="he", leaky=-0.5),
    LayerSpec("f4x2_2d_leaky", N=2, m=4, r=3, batch=3, C=40, K=75, X=(22, 29), pad=1,
              x_dist="normal", w_dist="he", leaky=0.2),
    LayerSpec("f4x3_3d_leaky", N=3, m=4, r=3, batch=1, C=20, K=24, X=(13, 11, 17), pad=1,
              x_dist="normal", w_dist="he", leaky=0.3),
    LayerSpec("f5x4_2d_leaky", N=2, m=5, r=4, batch=2, C=9, K=20, X=(23, 31), pad=0,
              x_dist="normal", w_dist="he", leaky=0.05),
    LayerSpec("f2x3_3d_parts_leaky", N=3, m=2, r=3, batch=2, C=512, K=192, X=(2, 7, 7), pad=1,
              x_dist="normal", w_dist="he", leaky=0.01),
]


@pytest.mark.parametrize("split", [True, False], ids=["split", "nosplit"])
@pytest.mark.parametrize("spec", LEAKY, ids=lambda s: s.name)
def test_leaky_relu_with_bias(spec, split):
    x, w = draw_layer(spec, seed=29)
    b = (np.random.default_rng(7).standard_normal(spec.K) * 0.5).astype(np.float32)
    y, plan = run_layer(spec, x, w, bias=b, guard=256, split=split)
    if not split:
        assert plan.desc["gemm_parts"] == 1
    assert np.any(y > 0) and (np.any(y < 0) if spec.leaky > 0 else True)
    check_full(spec, y, x, w, bias=b)
    y0, _ = run_layer(spec, x, w, guard=256, split=split)   # no bias
    check_full(spec, y0, x, w)


def test_bias_determinism_bitwise():
    # F(4^2): tail blocks split into parts, summed in order
    spec = SMALL[2]
    x, w = draw_layer(spec, seed=2)
    b = np.linspace(-1, 1, spec.K).astype(np.float32)
    y1, _ = run_layer(spec, x, w, bias=b, split=False)
    y2, _ = run_layer(spec, x, w, bias=b, split=False)
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))


@pytest.mark.parametrize("spec,points", [
    (SMALL[3], PAPER_F43_POINTS), (SMALL[2], PAPER_F43_POINTS),
    (SMALL[1], (0, 0.5, -0.5)), (SMALL[2], (0, -1, 1, 0.5, -2)),
], ids=["f43_3d_paper_pts", "f43_2d_paper_pts", "f23_half_pts", "f43_2d_other_pts"])
def test_caller_points(spec, points):
    x, w = draw_layer(spec, seed=5)
    y, plan = run_layer(spec, x, w, points=points)
    assert plan.desc["default_points"] == 0
    check_full(spec, y, x, w)


def test_searched_points_accuracy():
    """The point set wino_search_points picks for F(4^3, 3^3) (smallest error
    growth estimate) measures no less accurate than the paper's printed set,
    whose estimate is 27 times larger; every set stays within the m = 4 bar."""
    from paper_1611_06565_amd.wino import points_error_growth, search_points
    spec = LayerSpec("f4x3_3d_points", N=3, m=4, r=3, batch=1, C=32, K=24, X=(18, 17, 20), pad=1,
                     x_dist="uniform", w_dist="he")
    x, w = draw_layer(spec, seed=9)
    searched, g = search_points(3, 4, 3)
    errs = {}
    for name, pts in [("default", None), ("paper", PAPER_F43_POINTS), ("searched", searched)]:
        y, _ = run_layer(spec, x, w, points=pts)
        errs[name] = check_full(spec, y, x, w)["max"]
        log(f"  {name}: points {pts} growth {points_error_growth(3, 4, 3, pts):.1f} max err {errs[name]:.3e}")
    assert g < points_error_growth(3, 4, 3, PAPER_F43_POINTS)
    assert errs["searched"] <= errs["paper"]


@pytest.mark.parametrize("N,C", [(3, 16), (3, 5), (2, 16)])
def test_integer_inputs_bitwise_exact(N, C):
    spec = LayerSpec(f"int_f2x3_{N}d", N=N, m=2, r=3, batch=2, C=C, K=37,
                     X=(7, 9, 8)[:N] if N == 3 else (13, 11), pad=1,
                     x_dist="int2", w_dist="int2")
    x, w = draw_layer(spec, seed=3)
    y, _ = run_layer(spec, x, w)
    y_ref, _ = direct_blas(x, w, spec.pad)
    assert np.array_equal(y, y_ref.astype(np.float32))


def test_determinism_bitwise():
    spec = SMALL[1]
    x, w = draw_layer(spec, seed=2)
    y1, _ = run_layer(spec, x, w)
    y2, _ = run_layer(spec, x, w)
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))


@pytest.mark.parametrize("spec", [SMALL[1], SMALL[2], SMALL[3]], ids=lambda s: s.name)
def test_transform_stages_match_oracle(spec):
    """a2 and a3 on their own: U and V against the oracle's steps 2 and 3."""
    torch = require_gpu()
    from paper_1611_06565_amd.wino import Plan
    x, w = draw_layer(spec, seed=8)
    plan = Plan(spec.N, spec.m, spec.r, spec.C, spec.K, [spec.batch] + list(spec.X), pad=spec.pad)
    d = plan.desc
    U = plan.transform_filter(torch.from_numpy(w).cuda())
    ws = plan.transform_input(torch.from_numpy(x).cuda())
    torch.cuda.synchronize()
    nxi = d["n_xi"]
    Ug = plan.unpack_filter(U)
    Vg = plan.unpack_workspace(ws)
    Uo = o_filter(w, spec.m, spec.r).reshape(spec.K, spec.C, nxi).transpose(2, 1, 0)
    Vo = o_input(x, spec.m, spec.r, spec.pad).reshape(d["T"], spec.C, nxi).transpose(2, 1, 0)
    assert np.all(Ug[:, spec.C:, :] == 0) and np.all(Ug[:, :, spec.K:] == 0)
    assert np.all(Vg[:, spec.C:, :] == 0) and np.all(Vg[:, :, d["T"]:] == 0)
    scale_u = np.abs(Uo).max() + 1e-30
    assert np.abs(Ug[:, :spec.C, :spec.K] - Uo).max() <= 1e-6 * scale_u
    scale_v = np.abs(Vo).max() + 1e-30
    assert np.abs(Vg[:, :spec.C, :d["T"]] - Vo).max() <= 1e-6 * scale_v


def test_maxpool_matches_oracle():
    torch = require_gpu()
    from paper_1611_06565_amd.wino import maxpool3d
    rng = np.random.default_rng(1)
    # odd rows: the one-output-per-thread kernel; rows of a multiple of 4 with
    # a last-axis window of 2: the output-pair kernel (odd leading extents,
    # floors on every axis)
    for shape in [(2, 3, 5, 9, 7), (2, 3, 5, 9, 12), (1, 2, 3, 7, 8), (3, 1, 4, 6, 4)]:
        x = rng.standard_normal(shape).astype(np.float32)
        for win in [(1, 2, 2), (2, 2, 2), (2, 3, 1), (1, 1, 2), (3, 3, 2)]:
            if any(s // w < 1 for s, w in zip(shape[2:], win)):
                continue
            y = maxpool3d(torch.from_numpy(x).cuda(), win)
            torch.cuda.synchronize()
            assert np.array_equal(y.cpu().numpy(), maxpool(x, win)), (shape, win)


def test_small_c3d_stack_per_layer():
    """A narrow, small-volume copy of the C3D stack: every layer checked on
    every output against the oracle fed with the GPU's previous activations."""
    from workloads import StackSpec
    stack = StackSpec(name="c3d_small", batch=1, C_in=3, X=(16, 32, 32),
                      widths=(8, 16, 16, 16, 32, 32, 32, 32), pools=C3D_STACK.pools,
                      m=2, x_dist="uniform")
    _run_stack(stack, seed=4, full=True)


def _run_stack(stack, seed, full, ms=None):
    """Run the stack layer by layer (ms: the output tile of each layer), each
    layer's output checked against the oracle fed with the GPU's input."""
    torch = require_gpu()
    from paper_1611_06565_amd.wino import Plan, maxpool3d
    x, ws = draw_stack(stack, seed)
    cur = torch.from_numpy(x).cuda()
    for i, ((spec, pool), w) in enumerate(zip(stack.layers(), ws)):
        if ms is not None:
            spec = spec.with_(m=ms[i])
        log(f"[gpu] {spec.name} C={spec.C} K={spec.K} X={spec.X} m={spec.m}")
        plan = Plan(3, spec.m, 3, spec.C, spec.K, [spec.batch] + list(spec.X), pad=1, relu=True)
        U = plan.transform_filter(torch.from_numpy(w).cuda())
        y = plan.forward(cur, U)
        torch.cuda.synchronize()
        xin = cur.cpu().numpy()
        yh = y.cpu().numpy()
        if full:
            check_full(spec, yh, xin, w)
        else:
            check_sampled(spec, yh, xin, w, n=3000, seed=seed)
        if pool is not None:
            y = maxpool3d(y, pool.window)
            torch.cuda.synchronize()
            assert np.array_equal(y.cpu().numpy(), maxpool(yh, pool.window))
        cur = y
        del plan, U
    return cur


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_full_size_configs_full_output(cfg):
    spec = CONFIGS[cfg]
    x, w = draw_layer(spec, seed=cfg)
    y, plan = run_layer(spec, x, w)
    assert y.shape == (spec.batch, spec.K) + spec.out_spatial
    assert np.all(np.isfinite(y))
    assert plan.desc["fused"] == (1 if cfg == 4 else 0)
    check_full(spec, y, x, w)


def test_full_size_config4_two_stage_full_output():
    """The F(4^3) volume layer through V in memory (WINO_NO_FUSE)."""
    spec = CONFIGS[4]
    x, w = draw_layer(spec, seed=4)
    y, plan = run_layer(spec, x, w, fuse=False)
    assert plan.desc["fused"] == 0
    check_full(spec, y, x, w)


@pytest.mark.parametrize("cfg", [2, 3])
def test_full_size_bias_full_output(cfg):
    """The bench layers with a bias: whole blocks and split-tail parts in one launch."""
    spec = CONFIGS[cfg]
    x, w = draw_layer(spec, seed=cfg + 20)
    b = np.random.default_rng(cfg).standard_normal(spec.K).astype(np.float32)
    y, _ = run_layer(spec, x, w, bias=b)
    assert np.all(np.isfinite(y))
    check_full(spec, y, x, w, bias=b)


@pytest.mark.parametrize("cfg,slope", [(2, 0.1), (3, -0.25), (4, 0.2)])
def test_full_size_bias_leaky_full_output(cfg, slope):
    """The bench layers with a bias and a leaky ReLU as eq. (2)'s f, on every
    product kernel (m = 2, F(4^2), F(4^3))."""
    spec = CONFIGS[cfg].with_(leaky=slope, x_dist="normal")
    x, w = draw_layer(spec, seed=cfg + 40)
    b = (0.5 * np.random.default_rng(cfg + 1).standard_normal(spec.K)).astype(np.float32)
    y, _ = run_layer(spec, x, w, bias=b)
    assert np.all(np.isfinite(y))
    check_full(spec, y, x, w, bias=b)


def test_full_size_fig4_layer_full_output():
    """First layer of the paper's 2-D benchmark stand-in (F(5^2, 4^2), 224 x 224,
    C = K = 32) at batch 20."""
    spec = fig4_layers(batch=20)[0]
    x, w = draw_layer(spec, seed=100)
    y, _ = run_layer(spec, x, w)
    assert y.shape == (20, 32, 221, 221)
    assert np.all(np.isfinite(y))
    check_full(spec, y, x, w)


def test_full_size_c3d_stack_mixed_tiles_full_output():
    """The stack with F(4^3) on conv1-conv4 (conv1, 64 kernels, through the
    fused kernel with its 3 channels in one 8-channel chunk; conv2-conv4 in
    two stages) and F(2^3) on conv5-conv8, the per-layer choice that
    bench.py --stack-tiles times; every layer on every output, at its own
    tile's bar."""
    out = _run_stack(C3D_STACK, seed=6, full=True, ms=(4, 4, 4, 4, 2, 2, 2, 2))
    assert tuple(out.shape) == (4, 512, 1, 3, 3)


def test_full_size_c3d_stack_full_output():
    """The C3D-style stack at full size, every layer compared on every output
    against the oracle fed with the GPU's previous activations."""
    out = _run_stack(C3D_STACK, seed=5, full=True)
    assert tuple(out.shape) == (4, 512, 1, 3, 3)
