"""Benchmark: one step = one full pass of the tuning hot path on one workload.

A step draws the exploration samples, measures each on the GPU, hands the best
to Droplet Search, runs it to convergence (or its trial budget), and re-times
the winner.  `value` is the GFLOP/s of the tuned kernel (median over the timed
steps); `ms_per_step` is the wall-clock of one tuning pass.  Inputs are
resident in HBM before the timed region starts.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload matmul_1024]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tuned conv2d/matmul GFLOP/s + % fp32 roofline; measurements to reach best"
PEAK_FP32_TFLOPS = 157.3      # MI355X published fp32 (vector and MFMA), dense
PEAK_HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="matmul_1024")
    ap.add_argument("--n-explore", type=int, default=300)
    ap.add_argument("--budget", type=int, default=100)
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum CPU time of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}); the tuning path runs on a "
              "single device and has no multi-GPU mode.", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import synthdata
    from synthdata import workloads as wl
    from paper_2406_20037_amd import _lib as L

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    op, shape = wl.SINGLE[args.workload]
    flops = wl.flops(op, shape)
    abytes = wl.algorithmic_bytes(op, shape)
    if op == wl.OP_CONV:
        x, w = synthdata.conv_inputs(shape, "uniform")
        N, C, H, W, K, R, S, st, pd = shape
        P = (H + 2 * pd - R) // st + 1
        Q = (W + 2 * pd - S) // st + 1
        n_out = N * K * P * Q
        desc = f"conv2d NCHW fp32 N={N} C={C} H=W={H} K={K} {R}x{S} stride {st} pad {pd}"
    else:
        x, w = synthdata.matmul_inputs(shape, "uniform")
        n_out = shape[0] * shape[1]
        desc = f"matmul fp32 row-major M={shape[0]} N={shape[1]} K={shape[2]}"
    xd = torch.from_numpy(x).cuda()
    wd = torch.from_numpy(w).cuda()
    yd = torch.empty(n_out, dtype=torch.float32, device="cuda:0")
    stream = torch.cuda.current_stream()
    space = L.Space(op, shape)
    io = L.make_io(xd, wd, yd, None, stream)
    info = L.ds_device_info()
    log(f"device {info}; workload {desc}")

    final_cfg = L.measure_cfg(repeat=31, min_repeat_ms=2.0, max_number=1000, check=0)

    def step(seed):
        cfg = L.tune_cfg(n_explore=args.n_explore, budget=args.budget, seed=seed)
        res, _ = L.ds_tune(space, cfg, io)
        m = L.ds_measure(res.best, io, final_cfg)
        return res, m

    base_seed = wl.sampler_seed(1 if op == wl.OP_MATMUL else 0)
    for i in range(args.warmup):
        res, m = step(base_seed + 100 + i)
        log(f"warmup {i}: {space.knobs(res.best)} {m.median_ms * 1e3:.2f} us")
    floor = L.ds_empty_kernel_floor(stream)
    log(f"empty-kernel floor {floor.median_ms * 1e3:.2f} us")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    results = []
    for i in range(args.steps):
        res, m = step(base_seed + i)
        results.append((res, m))
        log(f"step {i}: best {space.knobs(res.best)} median {m.median_ms * 1e3:.2f} us "
            f"({flops / (m.median_ms * 1e-3) / 1e9:.0f} GFLOP/s), explored "
            f"{res.n_explore_measured}, droplet {res.n_droplet_measured}, {res.wall_s:.1f} s")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    gfs = [flops / (m.median_ms * 1e-3) / 1e9 for _, m in results]
    order = sorted(range(len(gfs)), key=lambda i: gfs[i])
    mid = order[len(order) // 2]
    res, m = results[mid]
    value = gfs[mid]
    avg_ms = m.mean_ms
    knobs = space.knobs(res.best)
    uses_mfma = bool(knobs.get("mfma", 0))
    achieved_tflops = flops / (avg_ms * 1e-3) / 1e12
    kname = kernel_name(op, knobs, space.geometry(res.best.index()))
    roofline = {
        "bound": "mfma" if uses_mfma else "alu",
        "achieved": round(achieved_tflops, 3),
        "peak": PEAK_FP32_TFLOPS,
        "unit": "TFLOP/s",
        "frac": round(achieved_tflops / PEAK_FP32_TFLOPS, 4),
        "traffic": measured_traffic(kname),
        "kernel": kname,
        "avg_launch_us": round(avg_ms * 1e3, 3),
        "algorithmic_flops": flops,
        "algorithmic_bytes": abytes,
    }

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(op, shape, x, w, flops, args.cpu_seconds, L, space, res.best, xd, wd, yd)

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall / max(1, args.steps) * 1e3, 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic: SplitMix64 U[-1,1) inputs, seeded",
        "config": {"workload": desc, "shape": list(shape), "n_explore": args.n_explore,
                   "droplet_budget": args.budget},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "tuning": {
            "best_schedule": knobs,
            "best_median_us": round(m.median_ms * 1e3, 3),
            "n_explore_measured": res.n_explore_measured,
            "n_droplet_measured": res.n_droplet_measured,
            "n_measured_total": res.n_explore_measured + res.n_droplet_measured,
            "n_failed": res.n_failed,
            "droplet_moves": res.n_moves,
            "seed_point_us": round(res.seed_ms * 1e3, 3),
            "tuning_wall_s": round(res.wall_s, 2),
            "explore_s": round(res.explore_s, 2),
            "droplet_s": round(res.droplet_s, 2),
            "per_step_gflops": [round(g, 1) for g in gfs],
            "empty_kernel_floor_us": round(floor.median_ms * 1e3, 3),
            "device": info,
        },
    }
    print(json.dumps(out), flush=True)
    return 0


def measured_traffic(kname):
    """HBM bytes per launch of this kernel instance from the committed rocprofv3
    counter runs (FETCH_SIZE and WRITE_SIZE, each scaled by the same counter on a
    copy of known size), or None when that instance was not profiled or its
    sources changed since."""
    from paper_2406_20037_amd.prof_summary import source_hash
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        data = json.load(fh)
    e = data.get(kname)
    if not e or e.get("source_sha256") != source_hash(kname):
        return None
    return int(round(e["read_bytes"] + e["write_bytes"]))


def kernel_name(op, knobs, geom):
    """Template instance the schedule selects (as rocprofv3 lists it)."""
    if op == 2:
        if knobs["mfma"]:
            return (f"mm_mfma<{geom['t0']}, {geom['t1']}, {knobs['bk']}, {geom['unroll_eff']}, "
                    f"{knobs['dbuf']}>")
        return (f"mm_valu<{geom['t0']}, {geom['t1']}, {knobs['bk']}, {geom['unroll_eff']}, "
                f"{knobs['dbuf']}>")
    fam = "conv_mfma" if knobs["mfma"] else "conv_valu"
    return f"{fam}<{geom['t0']}, {geom['t1']}, {geom['unroll_eff']}, {knobs['lds']}>"


def cpu_baseline(op, shape, x, w, flops, min_seconds, L, space, best, xd, wd, yd):
    """The fp64 oracle on the host cores, repeated until min_seconds elapse."""
    import numpy as np
    import torch

    from oracle import kernels as ok

    threads = ok.num_threads()
    runs, t = 0, 0.0
    ref = None
    while runs == 0 or t < min_seconds:
        t0 = time.perf_counter()
        ref = ok.conv2d_f64(x, w, shape) if op == 1 else ok.matmul_f64(x, w)
        t += time.perf_counter() - t0
        runs += 1
    L.kernel_run(op, best, xd, wd, yd)
    torch.cuda.synchronize()
    y = yd.cpu().numpy().astype(np.float64)
    rel = float(np.abs(y - ref.ravel()).max() / np.abs(ref).max())
    return {
        "value": round(flops * runs / t / 1e9, 2),
        "unit": "GFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"the full workload, {runs} run(s) in {t:.1f} s (fp64 accumulation, OpenMP)",
        "tuned_kernel_max_rel_err": rel,
    }


if __name__ == "__main__":
    sys.exit(main())
