#!/usr/bin/env python3
"""Throughput of the N-D Winograd forward on one MI355X.

Workload: the F(2^3, 3^3) video layer, batch 8, C = 64 -> K = 128, 16x56x56,
3x3x3 kernels, pad 1, fp32, inputs ReLU(N(0,1)) and He-normal weights from a
seed (synthetic stand-ins for C3D activations and weights).

One step is the whole hot path over the batch: kernel transform (a2), input
transform (a3) and the batched fp32-MFMA GEMM with the fused inverse
transform (a4 + a5).  Transform synthesis (a1) happens once, at plan time.
Inputs are resident in HBM before timing starts.  The metric is effective
TFLOP/s: direct-convolution FLOPs 2*n*K*C*27*prod(Y) per step time.

Prints one JSON line.  Per-stage durations come from HIP events recorded on
the stream the kernels run on; the roofline object reports the dominant
kernel against the MI355X fp32 MFMA peak.
"""
import argparse
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_MFMA = 157.3      # TFLOP/s, MI355X dense fp32 matrix
PEAK_HBM = 8000.0           # GB/s, MI355X HBM3E
PROFILE_DIR = os.path.join(ROOT, "profiles")
CSRC = "paper_1611_06565_amd/csrc/"
_COMMON = ["kernels.hpp", "transforms.hpp", "synth.hpp", "layout.hpp", "launch.hpp", "plan.hpp"]
# the sources that define each kernel family's code (a profile stays valid
# while they and the plan's launch geometry are unchanged)
FAMILY_SOURCES = {
    "m2": _COMMON + ["gemm_acc.hpp", "sizes_m2.hip"],
    "f42": _COMMON + ["gemm_acc.hpp", "gemm_acc4.hpp", "sizes_f42.hip"],
    "f43": _COMMON + ["sizes_f43.hip"],
    "f43fused": _COMMON + ["fused43.hpp", "fused_f43.hip"],
    "ax": _COMMON + ["aniso.hpp", "sizes_ax.hip"],
    "a8": _COMMON + ["sizes_f54.hip", "sizes_f45.hip", "sizes_f36.hip", "sizes_f32.hip"],
    "a8_3d": _COMMON + ["a8.hpp", "sizes_a8.hip"],
}
# normalised max-error bars per output-tile extent m (the same as the GPU tests')
TOL = {2: 1e-5, 3: 1e-4, 4: 1e-4, 5: 1e-4}


def family_of(desc):
    if desc.get("fused"):
        return "f43fused"
    tile = desc.get("tile", [])
    if desc["N"] == 3 and len(set(tile[:3])) > 1:
        return "ax"
    if desc["m"] == 2:
        return "m2"
    if (desc["N"], desc["m"], desc["r"]) == (2, 4, 3):
        return "f42"
    if (desc["N"], desc["m"], desc["r"]) == (3, 4, 3):
        return "f43"
    if desc["N"] == 3 and desc["n_xi"] == 512:
        return "a8_3d"
    return "a8"


def kernel_hash(desc=None):
    """sha256[:16] of a kernel family's sources and the plan's launch geometry
    (block sizes, padded sizes, tail split), or of every source without a plan."""
    h = hashlib.sha256()
    files = FAMILY_SOURCES[family_of(desc)] if desc is not None else sorted(
        {f for v in FAMILY_SOURCES.values() for f in v})
    for rel in files:
        with open(os.path.join(ROOT, CSRC, rel), "rb") as f:
            h.update(f.read())
    if desc is not None:
        geo = {k: desc[k] for k in ("T_pad", "C_pad", "K_pad", "block_tiles", "block_kernels", "gemm_parts",
                                    "gemm_tail_blocks", "fused", "tile")}
        h.update(json.dumps(geo, sort_keys=True).encode())
    return h.hexdigest()[:16]


def read_counters(expected_hash, config):
    """The GEMM kernel's counter summary (profiles/*_traffic.txt) taken on this
    workload with these kernel sources, as a dict, or {} if there is none."""
    for path in sorted(glob.glob(os.path.join(PROFILE_DIR, "*_traffic.txt"))):
        vals = {}
        with open(path) as f:
            for line in f:
                m = re.match(r"\s*(\w+)\s*[:=]\s*(\S+)", line)
                if m:
                    vals[m.group(1)] = m.group(2)
        if vals.get("kernel_sources_sha256_16") == expected_hash and vals.get("config") == str(config):
            return vals
    return {}


def read_traffic(expected_hash, config):
    """HBM bytes per launch of the GEMM kernel from the committed counter
    summary, or None if absent, taken on another workload or on different
    kernel sources."""
    try:
        return float(read_counters(expected_hash, config)["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def host_record():
    """The host the CPU baseline runs on: logical CPUs, CPU model, BLAS threads."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = None
    try:
        import threadpoolctl
        blas = max(int(i.get("num_threads", 1)) for i in threadpoolctl.threadpool_info()) or None
    except Exception:  # noqa: BLE001
        blas = None
    return {"os_cpu_count": os.cpu_count(), "cpu_model": model, "blas_threads": blas}


def cpu_baseline(spec, x, w, budget_s=10.0, winograd_budget_s=8.0):
    """Time the fp64 oracles on the host: the direct correlation (per-offset
    BLAS form) on whole samples of the batch until about budget_s seconds have
    elapsed, and the reference Winograd path (eq. 3-5 step by step) on one
    sample, cut along the first spatial axis to about winograd_budget_s."""
    import numpy as np

    from oracle.direct import direct_blas
    from oracle.winograd import winograd_forward
    from workloads import direct_flops
    host = host_record()
    threads = host["blas_threads"] or host["os_cpu_count"] or 1
    per_sample = direct_flops(spec) / spec.batch
    done, t_total = 0, 0.0
    while done < spec.batch and (done == 0 or t_total < budget_s):
        t0 = time.perf_counter()
        direct_blas(x[done:done + 1], w, spec.pad)
        t_total += time.perf_counter() - t0
        done += 1
    # reference Winograd: one sample, first axis cut to rows whose outputs
    # take about the budget (a slab of whole output rows, valid extent only)
    X0 = spec.X[0]
    rows, t_w, rows_done = max(1, 2 * spec.r), 0.0, 0
    while True:
        take = min(rows, X0)
        xs = x[:1, :, :take]
        t0 = time.perf_counter()
        winograd_forward(xs, w, spec.m, spec.r, pad=spec.pad)
        dt = time.perf_counter() - t0
        rows_done, t_w = take, dt
        if take == X0 or dt > winograd_budget_s / 4:
            break
        rows *= 2
    ys = [v + 2 * spec.pad - spec.r + 1 for v in (rows_done,) + tuple(spec.X[1:])]
    wino_flops = 2.0 * spec.K * spec.C * spec.r ** spec.N * float(np.prod(ys))
    return {
        "value": per_sample * done / t_total / 1e12,
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"fp64 direct correlation (per-offset BLAS form, with the |w||x| "
                   f"denominator) on {done} of {spec.batch} samples of the same layer, "
                   f"{t_total:.1f} s"),
        **host,
        "reference_winograd": {
            "value": wino_flops / t_w / 1e12, "unit": "TFLOP/s (direct FLOPs)",
            "sample": f"fp64 reference Winograd (tile, transforms, one product per element, inverse, "
                      f"stitch) on 1 sample cut to {rows_done} of {X0} rows of the first axis, {t_w:.1f} s"},
    }


def calib_copy(nbytes=1 << 30, reps=5):
    """A plain device copy of known size, for scaling HBM counters."""
    import torch
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calib_copy_bytes_each_way": nbytes, "reps": reps}), flush=True)


def bench_fig4(args):
    """The paper's 2-D benchmark (§4.4, Fig. 4) on synthetic stand-ins: a batch of
    224 x 224 images through three unpadded 4 x 4 layers of 32 channels and 32
    kernels with F(5^2, 4^2), transformed kernels cached; throughput in
    megavoxels (input pixels) per second, as the paper reports it."""
    import numpy as np
    import torch

    from paper_1611_06565_amd.wino import Plan
    from workloads import direct_flops, draw_layer, fig4_layers

    layers = fig4_layers(batch=args.fig4)
    plans, Us, wss, ys = [], [], [], []
    x0 = None
    for i, spec in enumerate(layers):
        x, w = draw_layer(spec, seed=100 + i)
        if i == 0:
            x0 = torch.from_numpy(x).cuda()
        plan = Plan(spec.N, spec.m, spec.r, spec.C, spec.K, [spec.batch] + list(spec.X), pad=spec.pad)
        plans.append(plan)
        Us.append(plan.transform_filter(torch.from_numpy(w).cuda()))
        wss.append(plan.new_workspace())
        ys.append(plan.new_output())
    torch.cuda.synchronize()

    def step(ev=None):
        src = x0
        for i, plan in enumerate(plans):
            if ev is not None:
                ev[2 * i].record()
            plan.transform_input(src, wss[i])
            if ev is not None:
                ev[2 * i + 1].record()
            plan.gemm_inverse(wss[i], Us[i], ys[i])
            src = ys[i]
        if ev is not None:
            ev[2 * len(plans)].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    nev = 2 * len(plans) + 1
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nev)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    st = np.array([[e[j].elapsed_time(e[j + 1]) for j in range(nev - 1)] for e in evs]).mean(axis=0)
    batch = layers[0].batch
    mvox = batch * layers[0].X[0] * layers[0].X[1] / (ms_step * 1e-3) / 1e6
    flops = sum(direct_flops(s) for s in layers)
    per_layer = []
    for i, (spec, plan) in enumerate(zip(layers, plans)):
        d = plan.desc
        g_bytes = 4.0 * (d["n_xi"] * d["T"] * spec.C + d["n_xi"] * spec.C * spec.K
                         + spec.batch * spec.K * float(np.prod(spec.out_spatial)))
        in_bytes = 4.0 * (spec.batch * spec.C * float(np.prod(spec.X)) + d["n_xi"] * d["T"] * spec.C)
        per_layer.append({"X": list(spec.X), "input_transform_us": float(st[2 * i]) * 1e3,
                          "gemm_inverse_us": float(st[2 * i + 1]) * 1e3,
                          "input_hbm_frac": in_bytes / (float(st[2 * i]) * 1e-3) / 1e9 / PEAK_HBM,
                          "gemm_hbm_frac": g_bytes / (float(st[2 * i + 1]) * 1e-3) / 1e9 / PEAK_HBM})
    out = {
        "metric": "MVox/s: 224x224 images through three 4x4 conv layers (C=K=32), F(5^2,4^2)",
        "value": mvox, "unit": "MVox/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"paper 2-D benchmark stand-in: batch {batch}, 224x224, 3 layers of 4x4, "
                               "C=K=32, unpadded, kernels transformed once", "batch": batch},
        "effective_tflops": flops / (ms_step * 1e-3) / 1e12,
        "layers": per_layer,
        "paper_cpu_MVox_s": 10.9,
    }
    print(json.dumps(out), flush=True)


def bench_stack(args):
    """The C3D-style stack (eight 3x3x3 pad-1 layers with fused ReLU, max-pools
    between them) forward with the transformed kernels cached: effective
    TFLOP/s over the direct FLOPs of all layers."""
    import numpy as np
    import torch

    from paper_1611_06565_amd.wino import Plan, maxpool3d
    from workloads import C3D_STACK, direct_flops, draw_stack

    x, ws = draw_stack(C3D_STACK, seed=5 if args.seed is None else args.seed)
    x0 = torch.from_numpy(x).cuda()
    # per-layer tiles: "2" F(2^3), "4" F(4^3), "244" per-axis (2, 4, 4), ...
    # default: F(4^3) while the output rows are at least 28 wide (conv1-4),
    # F(2^3) on the small late layers, where F(4^3)'s partial tiles waste work
    codes = (args.stack_tiles.split(",") if args.stack_tiles else
             ["4" if min(spec.out_spatial[1:]) >= 28 else "2" for spec, _ in C3D_STACK.layers()])
    if len(codes) != len(C3D_STACK.widths):
        raise SystemExit("--stack-tiles needs one code per layer")
    layers = []
    for (spec, pool), w, code in zip(C3D_STACK.layers(), ws, codes):
        tile = tuple(int(ch) for ch in code) if len(code) == 3 else None
        m = int(code) if tile is None else spec.m
        plan = Plan(3, m, 3, spec.C, spec.K, [spec.batch] + list(spec.X), pad=1, relu=True, tile=tile)
        U = plan.transform_filter(torch.from_numpy(w).cuda())
        wsp = plan.new_workspace()
        y = plan.new_output()
        py = None
        if pool is not None:
            Y = spec.out_spatial
            py = torch.empty((spec.batch, spec.K) + tuple(yy // p for yy, p in zip(Y, pool.window)),
                             dtype=torch.float32, device="cuda")
        # the pool rides on the product's epilogue (wino_forward_pool): F(4^3)
        # with windows (1,2,2) and (2,2,2), F(2^3) with (2,2,2)
        tile_now = tuple(plan.desc["tile"])
        fpool = (pool is not None and not args.no_fuse_pool
                 and ((tile_now == (4, 4, 4) and tuple(pool.window) in ((1, 2, 2), (2, 2, 2)))
                      or (tile_now == (2, 2, 2) and tuple(pool.window) == (2, 2, 2))))
        layers.append((spec, pool, plan, U, wsp, y, py, fpool))
    torch.cuda.synchronize()
    fused_pools = [L[0].name for L in layers if L[7]]
    pool_note = ("; max-pool in the product's epilogue on " + ",".join(fused_pools)) if fused_pools else ""

    def step(ev=None):
        cur = x0
        for i, (spec, pool, plan, U, wsp, y, py, fpool) in enumerate(layers):
            if ev is not None:
                ev[i].record()
            if fpool:
                plan.forward_pool(cur, U, pool.window, y=py, workspace=wsp)
                cur = py
                continue
            plan.forward(cur, U, y=y, workspace=wsp)
            cur = y
            if pool is not None:
                maxpool3d(y, pool.window, py)
                cur = py
        if ev is not None:
            ev[len(layers)].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if args.graph:
        # the whole step (19 launches) captured once as a HIP graph and replayed
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            step()
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            g.replay()
        torch.cuda.synchronize()
        ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
        flops = [direct_flops(spec) for spec, *_ in layers]
        print(json.dumps({
            "metric": "effective TFLOP/s of the C3D-style 3-D stack forward (direct FLOPs; kernels transformed once)",
            "value": sum(flops) / (ms_step * 1e-3) / 1e12, "unit": "TFLOP/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
            "config": {"workload": "C3D-style stack: batch 4, 3x16x112x112, eight 3x3x3 pad-1 layers "
                                   "(64, 128, 256, 256, 512 x4), ReLU, max-pools; tiles per layer " + ",".join(codes)
                                   + pool_note + "; one HIP graph per step"}}), flush=True)
        return
    nev = len(layers) + 1
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nev)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    st = np.array([[e[j].elapsed_time(e[j + 1]) for j in range(nev - 1)] for e in evs]).mean(axis=0)
    flops = [direct_flops(spec) for spec, *_ in layers]
    out = {
        "metric": "effective TFLOP/s of the C3D-style 3-D stack forward (direct FLOPs; kernels transformed once)",
        "value": sum(flops) / (ms_step * 1e-3) / 1e12, "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "C3D-style stack: batch 4, 3x16x112x112, eight 3x3x3 pad-1 layers "
                               "(64, 128, 256, 256, 512 x4), ReLU, max-pools; tiles per layer " + ",".join(codes)
                               + pool_note},
        "layers": [{"name": spec.name, "C": spec.C, "K": spec.K, "X": list(spec.X), "pool": bool(pool),
                    "tile": plan.desc["tile"],
                    "ms": float(st[i]), "tflops": flops[i] / (float(st[i]) * 1e-3) / 1e12,
                    "pool_fused": bool(fpool)}
                   for i, (spec, pool, plan, U, wsp, y, py, fpool) in enumerate(layers)],
    }
    print(json.dumps(out), flush=True)


def bench_wgrad(args):
    """The weight gradient of one layer (wino_weight_gradient: input
    transform, output-gradient transform, the product over the tiles and
    A'^T): effective TFLOP/s over the direct FLOPs of the same layer."""
    import numpy as np
    import torch

    from paper_1611_06565_amd.wino import Plan
    from workloads import CONFIGS, direct_flops, draw_layer

    spec = CONFIGS[args.config]
    seed = args.config if args.seed is None else args.seed
    x, _ = draw_layer(spec, seed=seed)
    plan = Plan(spec.N, spec.m, spec.r, spec.C, spec.K, [spec.batch] + list(spec.X), pad=spec.pad)
    d = plan.desc
    dy = np.random.default_rng(seed + 200).standard_normal(plan.output_shape, dtype=np.float32)
    xd, dyd = torch.from_numpy(x).cuda(), torch.from_numpy(dy).cuda()
    ws = torch.empty(plan.weight_gradient_workspace_bytes // 4, dtype=torch.float32, device="cuda")
    dw = torch.empty(plan.weight_shape, dtype=torch.float32, device="cuda")
    for _ in range(args.warmup):
        plan.weight_gradient(xd, dyd, dw, ws)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t0 = time.perf_counter()
    ev[0].record()
    for i in range(args.steps):
        plan.weight_gradient(xd, dyd, dw, ws)
        ev[i + 1].record()
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    ev_ms = float(np.mean([ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)]))
    flops = direct_flops(spec)
    gemm_flops = 2.0 * d["n_xi"] * d["T"] * spec.C * spec.K
    check = None
    if not args.no_check:
        from oracle.metric import normalised_error
        from oracle.wgrad import direct_wgrad
        ref, den = direct_wgrad(x, dy, spec.r, spec.pad)
        check = normalised_error(dw.cpu().numpy(), ref, den)["max"]
    out = {
        "metric": "effective TFLOP/s of a conv layer's weight gradient (direct FLOPs)",
        "value": flops / (ms_step * 1e-3) / 1e12, "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "weight gradient of F(%d^%d,3^%d) %d-D conv layer: batch %d, C=%d, K=%d, %s, pad %d"
                               % (spec.m, spec.N, spec.N, spec.N, spec.batch, spec.C, spec.K,
                                  "x".join(str(v) for v in spec.X), spec.pad)},
        "call_ms_events": ev_ms,
        # the product over the tiles, 2 * alpha^N * T * C * K FLOP, over the whole call
        "gemm_tflops_over_call": gemm_flops / (ev_ms * 1e-3) / 1e12,
        "max_normalised_error": check,
    }
    print(json.dumps(out), flush=True)
    if check is not None and not check <= 1e-4:
        print(f"bench.py: weight gradient misses the oracle by {check:.3e}", file=sys.stderr)
        sys.exit(3)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--config", type=int, default=2, choices=[1, 2, 3, 4, 5],
                    help="layer family (default 2, the F(2^3,3^3) C=64 K=128 video layer; "
                         "5 = the C3D-style stack)")
    ap.add_argument("--graph", action="store_true",
                    help="with --config 5: replay each step as one captured HIP graph")
    ap.add_argument("--wgrad", action="store_true",
                    help="time the layer's weight gradient dw from x and dy instead of its forward")
    ap.add_argument("--adjoint", action="store_true",
                    help="time the layer's data gradient dx = adjoint(dy) instead of its forward")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-check", action="store_true")
    ap.add_argument("--no-cold", action="store_true", help="skip the cold-cache repetitions")
    ap.add_argument("--stack-tiles", default=None, metavar="CODES",
                    help="with --config 5: per-layer tiles, e.g. 2,2,244,244,244,244,2,2 (default F(4^3) on layers "
                         "with output rows of 28 or more, F(2^3) after them: 4,4,4,4,2,2,2,2)")
    ap.add_argument("--tile", default=None, metavar="M0,M1,M2",
                    help="per-axis output tiles of the chosen 3-D layer, e.g. 2,4,4")
    ap.add_argument("--size", default=None, metavar="M,R",
                    help="another tile and kernel size on the chosen layer's shape, e.g. 5,4 for F(5^3,4^3) "
                         "(pad (r - 1) // 2)")
    ap.add_argument("--no-fuse", action="store_true",
                    help="keep an F(4^3) forward in two stages (input transform to V, then the product)")
    ap.add_argument("--no-fuse-pool", action="store_true",
                    help="with --config 5: run every max-pool as its own kernel (not in the product's epilogue)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="only run a 1 GiB device copy (for HBM counter scaling)")
    ap.add_argument("--fig4", type=int, default=0, metavar="BATCH",
                    help="run the paper's 2-D benchmark stand-in (three 4x4 layers, 224x224) at this batch")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build runs the layer on a single MI355X "
              "(sharding the batch or slabs of the volume across GPUs is designed but not built); "
              "run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    if args.calib_copy:
        calib_copy()
        return
    if args.fig4:
        bench_fig4(args)
        return
    if args.config == 5:
        bench_stack(args)
        return
    if args.wgrad:
        bench_wgrad(args)
        return

    from paper_1611_06565_amd.wino import Plan
    from workloads import CONFIGS, direct_flops, draw_layer

    spec = CONFIGS[args.config]
    if args.size:
        # another (m, r) on the same layer shape; pad (r - 1) // 2 per axis
        m_, r_ = (int(v) for v in args.size.split(","))
        spec = spec.with_(m=m_, r=r_, pad=(r_ - 1) // 2, name=f"{spec.name}_f{m_}x{r_}")
    seed = args.config if args.seed is None else args.seed
    x, w = draw_layer(spec, seed=seed)
    tile = tuple(int(v) for v in args.tile.split(",")) if args.tile else None
    plan = Plan(spec.N, spec.m, spec.r, spec.C, spec.K, [spec.batch] + list(spec.X),
                pad=spec.pad, relu=spec.relu, fuse=not args.no_fuse, tile=tile)
    transform_filter = plan.transform_filter
    if args.adjoint:
        # the data gradient: dy of the layer's output shape through the
        # adjoint plan, kernels flipped and transposed by its filter transform
        plan = plan.adjoint()
        transform_filter = plan.transform_filter_adjoint
        x = np.random.default_rng(seed + 100).standard_normal(plan.input_shape, dtype=np.float32)
    d = plan.desc
    xd = torch.from_numpy(x).cuda()
    wd = torch.from_numpy(w).cuda()
    U = plan.new_filter()
    ws = plan.new_workspace()
    y = plan.new_output()
    torch.cuda.synchronize()

    fused = bool(d["fused"])

    # One step: kernel transform, input transform, then the batched GEMM with
    # the inverse transform (the two calls wino_forward makes), each timed.
    # A fused plan (F(4^3), few kernels) runs the last two in one kernel: its
    # stage is recorded as the GEMM stage and the input stage is empty.
    def step(ev=None):
        if ev is not None:
            ev[0].record()
        transform_filter(wd, U)
        if ev is not None:
            ev[1].record()
        if not fused:
            plan.transform_input(xd, ws)
        if ev is not None:
            ev[2].record()
        if fused:
            plan.forward(xd, U, y=y)
        else:
            plan.gemm_inverse(ws, U, y)
        if ev is not None:
            ev[3].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    st = np.array([[e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2]), e[2].elapsed_time(e[3])]
                   for e in evs])
    filt_ms, inp_ms, gemm_ms = (float(v) for v in st.mean(axis=0))
    fwd_ms = inp_ms + gemm_ms

    # Cold-cache variant (outside the timed region above): a 1 GiB read
    # between repetitions evicts the L2s and the 256 MB memory-side cache, so
    # the stages read x, V and U from HBM.  A read, not a write: written
    # lines would still be dirty in the caches and their write-back would
    # compete with the next stage's traffic.
    cold = None
    if not args.no_cold:
        flush = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        sink = flush.sum()
        cev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
        for i in range(args.steps):
            sink += flush.sum()
            step(cev[i])
        torch.cuda.synchronize()
        cst = np.array([[e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2]), e[2].elapsed_time(e[3])]
                        for e in cev]).mean(axis=0)
        cold = ({"filter_transform": float(cst[0]), "fused_forward": float(cst[2])} if fused else
                {"filter_transform": float(cst[0]), "input_transform": float(cst[1]),
                 "gemm_inverse": float(cst[2])})
        del flush, sink

    flops = direct_flops(spec)
    nxi = d["n_xi"]
    C, K = plan.C, plan.K                    # swapped for the data gradient
    gemm_flops = 2.0 * nxi * d["T"] * C * K
    in_bytes = 4.0 * (float(np.prod(plan.input_shape)) + nxi * d["T"] * C)
    # The GEMM's algorithmic bytes: V read once, U read once, y written once.
    # Below the ridge point (peak FLOP/s over peak bytes/s) it is bound by HBM.
    gemm_bytes = 4.0 * (nxi * d["T"] * C + nxi * C * K + float(np.prod(plan.output_shape)))
    if fused:
        # the fused kernel reads x (not V), U, and writes y
        gemm_bytes = 4.0 * (float(np.prod(plan.input_shape)) + nxi * C * K + float(np.prod(plan.output_shape)))
    hbm_bound = gemm_flops / gemm_bytes < PEAK_FP32_MFMA * 1e12 / (PEAK_HBM * 1e9)
    if hbm_bound:
        achieved = gemm_bytes / (gemm_ms * 1e-3) / 1e9
    else:
        achieved = gemm_flops / (gemm_ms * 1e-3) / 1e12
    prof_key = (f"{args.config}" + ("-adjoint" if args.adjoint else "") + ("-no-fuse" if args.no_fuse else "")
                + (f"-tile{args.tile}" if args.tile else "") + (f"-size{args.size}" if args.size else ""))
    khash = kernel_hash(d)
    counters = read_counters(khash, prof_key)
    traffic = read_traffic(khash, prof_key)
    try:
        mfma_counted = float(counters["mfma_flops_per_launch"])
    except (KeyError, ValueError):
        mfma_counted = None

    check = None
    bar = TOL[max(tile)] if tile else TOL[spec.m]
    if not args.no_check:
        from oracle.direct import direct_sampled
        from oracle.metric import normalised_error
        rng = np.random.default_rng(0)
        yh = y.cpu().numpy()
        coords = np.stack([rng.integers(0, s, size=2000) for s in yh.shape], axis=1)
        if args.adjoint:
            from oracle.adjoint import direct_adjoint_sampled
            ys, dens = direct_adjoint_sampled(x, w, spec.pad, coords)
        else:
            ys, dens = direct_sampled(x, w, spec.pad, coords)
        check = normalised_error(yh[tuple(coords.T)], ys, dens)["max"]

    extra = {}
    if fused:
        extra["fused_forward_hbm"] = {
            "algorithmic_bytes": gemm_bytes, "achieved_GBps": gemm_bytes / (gemm_ms * 1e-3) / 1e9,
            "peak_GBps": PEAK_HBM, "frac": gemm_bytes / (gemm_ms * 1e-3) / 1e9 / PEAK_HBM}
    else:
        extra["input_transform_hbm"] = {"achieved_GBps": in_bytes / (inp_ms * 1e-3) / 1e9,
                                        "peak_GBps": PEAK_HBM,
                                        "frac": in_bytes / (inp_ms * 1e-3) / 1e9 / PEAK_HBM}
    if cold is not None:
        c_in, c_g = (0.0, cold["fused_forward"]) if fused else (cold["input_transform"], cold["gemm_inverse"])
        extra["cold_cache"] = {
            "stages_ms": cold,
            "forward_tflops": flops / ((c_in + c_g) * 1e-3) / 1e12,
            "input_transform_hbm_frac": (in_bytes / (c_in * 1e-3) / 1e9 / PEAK_HBM) if not fused else None,
            "gemm_frac": ((gemm_bytes / (c_g * 1e-3) / 1e9 / PEAK_HBM) if hbm_bound
                          else (gemm_flops / (c_g * 1e-3) / 1e12 / PEAK_FP32_MFMA)),
            "gemm_bound": "hbm" if hbm_bound else "mfma",
            "flush": "1 GiB device read between repetitions",
        }
    if check is not None:
        extra["parity"] = {"max_normalised_error_sampled": check, "tolerance": bar,
                           "ok": bool(check <= bar)}
    out = {
        "metric": ("effective TFLOP/s of a conv layer's data gradient (direct FLOPs); % fp32 MFMA / HBM peak"
                   if args.adjoint else
                   "effective TFLOP/s per 3D conv layer (direct FLOPs); % fp32 MFMA / HBM peak"),
        "value": flops / (ms_step * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": ("data gradient (adjoint plan: C and K swapped, pads r-1-pad) of " if args.adjoint
                         else "") + ("F(%s,3^%d) per-axis tiles " % ("x".join(str(v) for v in tile), spec.N)
                                     if tile else "F(%d^%d,%d^%d) " % (spec.m, spec.N, spec.r, spec.N)) +
                        "%d-D conv layer: batch %d, C=%d, K=%d, %s, %s, pad %d" % (
                spec.N, spec.batch, spec.C, spec.K,
                "x".join(str(v) for v in spec.X), "x".join([str(spec.r)] * spec.N), spec.pad),
            "N": spec.N, "m": spec.m, "r": spec.r, "batch": spec.batch, "C": spec.C, "K": spec.K,
            "X": list(spec.X), "pad": spec.pad,
            "points": ",".join(["0", "1", "-1", "2", "-2", "1/2", "-1/2"][:spec.m + spec.r - 2] + ["inf"]),
            "seed": seed,
            "tile": list(tile) if tile else [spec.m] * spec.N,
            "tiles": d["T"], "direct_gflop_per_step": flops / 1e9,
        },
        "roofline": {
            "kernel": ("k_fused43 (input transform in LDS, batched fp32-MFMA GEMM, fused inverse transform; "
                       "V never in memory)" if fused else
                       "k_gemm_ax (batched fp32-MFMA GEMM, per-axis inverse transform)" if tile else
                       "k_gemm_a8 (batched fp32-MFMA GEMM over each first-axis plane of the 512 elements, "
                       "inverse transform accumulated plane by plane)" if spec.N == 3 and d["n_xi"] == 512 else
                       "k_gemm_acc + k_part_reduce (batched fp32-MFMA GEMM, inverse transform accumulated "
                       "per pass; the %d tail blocks in %d parts each, their partial outputs summed in order)"
                       % (d["gemm_tail_blocks"], d["gemm_parts"])
                       if spec.m == 2 and d["gemm_parts"] > 1 else
                       "k_gemm_acc (batched fp32-MFMA GEMM, inverse transform accumulated per pass)"
                       if spec.m == 2 else
                       "k_gemm_acc4 + k_part_reduce (batched fp32-MFMA GEMM, inverse transform accumulated "
                       "per pass; the %d tail blocks in %d parts each, their partial outputs summed in order)"
                       % (d["gemm_tail_blocks"], d["gemm_parts"])
                       if (spec.N, spec.m, spec.r) == (2, 4, 3) and d["gemm_parts"] > 1 else
                       "k_gemm_acc4 (batched fp32-MFMA GEMM, inverse transform accumulated per pass)"
                       if (spec.N, spec.m, spec.r) == (2, 4, 3) else
                       "k_gemm_inv (batched fp32-MFMA GEMM + fused inverse transform)"),
            "bound": "hbm" if hbm_bound else "mfma",
            "achieved": achieved,
            "peak": PEAK_HBM if hbm_bound else PEAK_FP32_MFMA,
            "unit": "GB/s" if hbm_bound else "TFLOP/s",
            "frac": achieved / (PEAK_HBM if hbm_bound else PEAK_FP32_MFMA),
            "traffic": traffic,
            "algorithmic": ("4*(alpha^N*T*C + alpha^N*C*K + n*K*prod(Y)) = %.4g bytes per launch" % gemm_bytes
                            if hbm_bound else "2*alpha^N*T*C*K = %.4g FLOP per launch" % gemm_flops),
            "gemm_tflops": gemm_flops / (gemm_ms * 1e-3) / 1e12,
            # MFMA work counted by rocprofv3 (SQ_INSTS_VALU_MFMA_MOPS_F32 x 512)
            # on these kernel sources, and the MFMA fraction it gives here
            "mfma_flops_counted": mfma_counted,
            "mfma_frac_counted": (mfma_counted / (gemm_ms * 1e-3) / 1e12 / PEAK_FP32_MFMA
                                  if mfma_counted is not None else None),
        },
        "stages_ms": ({"filter_transform": filt_ms, "fused_forward": gemm_ms} if fused else
                      {"filter_transform": filt_ms, "input_transform": inp_ms, "gemm_inverse": gemm_ms}),
        "forward_U_cached_tflops": flops / (fwd_ms * 1e-3) / 1e12,
        "max_normalised_error_sampled": check,
        "kernel_sources_sha256_16": khash,
    }
    out.update(extra)
    if not args.no_cpu_baseline and not args.adjoint:
        out["cpu_baseline"] = cpu_baseline(spec, x, w)
    print(json.dumps(out), flush=True)
    if check is not None and not check <= bar:
        print(f"bench.py: the sampled outputs miss the oracle by {check:.3e} "
              f"(bar {bar:.0e}): the throughput above is of a wrong result", file=sys.stderr)
        sys.exit(3)


if __name__ == "__main__":
    main()
