"""Helpers for the GPU parity tests: run a layer through the C ABI and compare
with the fp64 oracle on the same seeded inputs."""
import sys

import numpy as np

from oracle.direct import direct_blas, direct_sampled
from oracle.metric import normalised_error

# normalised max error per output-tile extent m: the stated bars for m = 2
# and 4; the other 2-D sizes (F(3,2), F(5,4), F(4,5), F(3,6)) take the m = 4
# bar (F(5,4)'s measured max errors are about 3e-6, a margin of 30 like F(4^3)'s)
TOL = {2: 1e-5, 3: 1e-4, 4: 1e-4, 5: 1e-4}


def tol(spec):
    """The bar of a layer: the m = 4 bar when any axis has a tile of 4 or more."""
    return TOL[max(spec.tile)] if spec.tile else TOL[spec.m]


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def require_gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    import paper_1611_06565_amd.wino as wino
    wino.lib()  # raises if the library is not built
    return torch


def run_layer(spec, x, w, points=None, guard=0, bias=None, split=True, fuse=True):
    """Plan, transform the filter and run the forward.  Returns (y numpy, plan).

    With guard > 0 the output is a view inside a larger buffer whose guard
    bands hold a sentinel; the bands are checked afterwards."""
    torch = require_gpu()
    from paper_1611_06565_amd.wino import Plan
    log(f"[gpu] {spec.name} N={spec.N} m={spec.m} C={spec.C} K={spec.K} X={spec.X} "
        f"batch={spec.batch} pad={spec.pad} points={points} split={split} fuse={fuse} relu={spec.relu} "
        f"leaky={spec.leaky} tile={spec.tile}")
    plan = Plan(spec.N, spec.m, spec.r, spec.C, spec.K, [spec.batch] + list(spec.X),
                pad=spec.pad, points=points, relu=spec.relu, split=split, leaky=spec.leaky, fuse=fuse,
                tile=spec.tile)
    xd = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    wd = torch.from_numpy(np.ascontiguousarray(w)).cuda()
    U = plan.transform_filter(wd)
    ws = plan.new_workspace()
    n_out = int(np.prod(plan.output_shape))
    if guard:
        buf = torch.full((n_out + 2 * guard,), 12345.5, dtype=torch.float32, device="cuda")
        y = buf[guard:guard + n_out].view(plan.output_shape)
    else:
        y = plan.new_output()
    bd = torch.from_numpy(np.ascontiguousarray(bias)).cuda() if bias is not None else None
    plan.forward(xd, U, y=y, workspace=ws, bias=bd)
    torch.cuda.synchronize()
    if guard:
        b = buf.cpu().numpy()
        assert np.all(b[:guard] == 12345.5) and np.all(b[-guard:] == 12345.5), "guard band written"
    return y.cpu().numpy(), plan


def check_full(spec, y, x, w, bias=None):
    y_ref, den = direct_blas(x, w, spec.pad, relu=spec.relu, bias=bias, leaky=spec.leaky)
    err = normalised_error(y, y_ref, den)
    log(f"  max err {err['max']:.3e} p99.99 {err['p9999']:.3e} at {err['argmax']} "
        f"clamped {err['clamped']}")
    assert err["nonfinite"] == 0
    assert err["max"] <= tol(spec), err
    return err


def sample_coords(shape, n, rng, edges=True):
    """n uniform output coordinates plus the corners of every axis."""
    coords = [rng.integers(0, s, size=n) for s in shape]
    out = np.stack(coords, axis=1)
    if edges:
        corners = []
        for b in (0, shape[0] - 1):
            for k in (0, shape[1] - 1):
                for lo in range(2 ** (len(shape) - 2)):
                    c = [b, k] + [(shape[2 + a] - 1) if (lo >> a) & 1 else 0
                                  for a in range(len(shape) - 2)]
                    corners.append(c)
        out = np.concatenate([out, np.array(corners)], axis=0)
    return out


def check_sampled(spec, y, x, w, n=4000, seed=0, bias=None):
    rng = np.random.default_rng(seed)
    coords = sample_coords(y.shape, n, rng)
    ys, dens = direct_sampled(x, w, spec.pad, coords, relu=spec.relu, bias=bias, leaky=spec.leaky)
    got = y[tuple(coords.T)]
    err = normalised_error(got, ys, dens)
    log(f"  sampled {len(coords)}: max err {err['max']:.3e} p99.99 {err['p9999']:.3e}")
    assert np.all(np.isfinite(y[tuple(coords.T)]))
    assert err["max"] <= tol(spec), err
    return err
