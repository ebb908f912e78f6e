"""Benchmark: one step = one full pass of the tuning hot path on one workload.

A step draws the exploration samples, measures each on the GPU, hands the best
to Droplet Search, runs it to convergence (or its trial budget), and re-times
the winner -- for every task of the workload (one task for a single kernel;
every distinct layer for a network, each with its own sampler seed).  `value`
is the GFLOP/s of the tuned kernels (for a network: total weighted flops over
total weighted tuned time), median over the timed steps; `ms_per_step` is the
wall-clock of one tuning pass.  Inputs are resident in HBM before the timed
region starts.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload matmul_1024]
    python bench.py --workload resnet50 --steps 1 --warmup 0 [--flush]
    python bench.py --workload vgg16 --layers 0-6 --steps 1 --warmup 0
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tuned conv2d/matmul GFLOP/s + % fp32 roofline; measurements to reach best"
PEAK_FP32_TFLOPS = 157.3      # MI355X published fp32 (vector and MFMA), dense
PEAK_HBM_GBS = 8000.0         # MI355X published HBM3E bandwidth

SINGLE_CONFIG = {"conv3x3_c64_56": 0, "matmul_1024": 1, "conv7x7_s2_c3_224": 2}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def workload_tasks(name, layers):
    """[(task name, op, shape, count, layer index)], input kind, config number."""
    from synthdata import workloads as wl
    if name in wl.SINGLE:
        op, shape = wl.SINGLE[name]
        return [(name, op, shape, 1, 0)], "uniform", SINGLE_CONFIG[name]
    if name == "resnet50":
        tasks, kind, cfg = wl.RESNET50, "he", 3
    elif name == "vgg16":
        tasks, kind, cfg = wl.VGG16, "he", 4
    else:
        raise SystemExit(f"unknown workload {name}")
    idx = list(range(len(tasks)))
    if layers:
        idx = []
        for part in layers.split(","):
            a, _, b = part.partition("-")
            idx += list(range(int(a), int(b or a) + 1))
    return [(tasks[i][0], tasks[i][1], tasks[i][2], tasks[i][3], i) for i in idx], kind, cfg


def describe(op, shape):
    if op == 1:
        N, C, H, W, K, R, S, st, pd = shape
        return f"conv2d NCHW fp32 N={N} C={C} H=W={H} K={K} {R}x{S} stride {st} pad {pd}"
    return f"matmul fp32 row-major M={shape[0]} N={shape[1]} K={shape[2]}"


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="matmul_1024",
                    help="matmul_1024 | conv3x3_c64_56 | conv7x7_s2_c3_224 | resnet50 | vgg16")
    ap.add_argument("--layers", default="", help="network workloads: task indices, e.g. 0-6,9")
    ap.add_argument("--n-explore", type=int, default=300)
    ap.add_argument("--budget", type=int, default=100)
    ap.add_argument("--flush", action="store_true",
                    help="also time each tuned kernel cold (512 MB written between launches)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum CPU time of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}); the tuning path runs on a "
              "single device and has no multi-GPU mode.", file=sys.stderr)
        return 2

    import torch

    import synthdata
    from synthdata import workloads as wl
    from paper_2406_20037_amd import _lib as L

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    tasks, kind, config = workload_tasks(args.workload, args.layers)
    single = args.workload in wl.SINGLE
    stream = torch.cuda.current_stream()
    info = L.ds_device_info()
    log(f"device {info}; workload {args.workload}: {len(tasks)} task(s)")

    # Inputs of every task, resident on the device before any timing.
    T = []
    for name, op, shape, count, layer in tasks:
        if op == wl.OP_CONV:
            x, w = synthdata.conv_inputs(shape, kind)
            P, Q = synthdata.conv_out_hw(shape[2], shape[3], shape[5], shape[6], shape[7], shape[8])
            n_out = shape[0] * shape[4] * P * Q
        else:
            x, w = synthdata.matmul_inputs(shape, kind)
            n_out = shape[0] * shape[1]
        xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
        yd = torch.empty(n_out, dtype=torch.float32, device="cuda:0")
        space = L.Space(op, shape)
        T.append(dict(name=name, op=op, shape=shape, count=count, layer=layer, x=x, w=w, xd=xd,
                      wd=wd, yd=yd, space=space, io=L.make_io(xd, wd, yd, None, stream),
                      flops=wl.flops(op, shape), bytes=wl.algorithmic_bytes(op, shape)))

    final_cfg = L.measure_cfg(repeat=31, min_repeat_ms=2.0, max_number=1000, check=0)

    def step(offset, tag):
        out = []
        for task in T:
            seed = wl.sampler_seed(config, task["layer"]) + offset
            cfg = L.tune_cfg(n_explore=args.n_explore, budget=args.budget, seed=seed)
            res, _ = L.ds_tune(task["space"], cfg, task["io"])
            m = L.ds_measure(res.best, task["io"], final_cfg)
            out.append((res, m))
            log(f"{tag} {task['name']}: best {task['space'].knobs(res.best)} "
                f"{m.median_ms * 1e3:.2f} us ({task['flops'] / (m.median_ms * 1e-3) / 1e9:.0f} "
                f"GFLOP/s), explored {res.n_explore_measured}, droplet {res.n_droplet_measured}, "
                f"{res.wall_s:.1f} s")
        return out

    for i in range(args.warmup):
        step(100 + i, f"warmup {i}")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    steps = []
    for i in range(args.steps):
        steps.append(step(i, f"step {i}"))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    floor = L.ds_empty_kernel_floor(stream)      # after the steps: the device is warm
    log(f"empty-kernel floor {floor.median_ms * 1e3:.2f} us")

    def network_gflops(st):
        tot_f = sum(task["count"] * task["flops"] for task in T)
        tot_t = sum(task["count"] * m.median_ms * 1e-3 for task, (_, m) in zip(T, st))
        return tot_f / tot_t / 1e9

    gfs = [network_gflops(st) for st in steps]
    order = sorted(range(len(gfs)), key=lambda i: gfs[i])
    chosen = steps[order[len(order) // 2]]
    value = gfs[order[len(order) // 2]]

    per_task = []
    for task, (res, m) in zip(T, chosen):
        knobs = task["space"].knobs(res.best)
        ai = task["flops"] / task["bytes"]
        hbm_bound = ai * PEAK_HBM_GBS * 1e9 < PEAK_FP32_TFLOPS * 1e12
        attainable = ai * PEAK_HBM_GBS * 1e9 if hbm_bound else PEAK_FP32_TFLOPS * 1e12
        achieved = task["flops"] / (m.median_ms * 1e-3)
        row = dict(name=task["name"], count=task["count"], shape=list(task["shape"]),
                   best_schedule=knobs,
                   kernel=kernel_name(task["op"], knobs, task["space"].geometry(res.best.index())),
                   best_us=round(m.median_ms * 1e3, 3), mean_us=round(m.mean_ms * 1e3, 3),
                   gflops=round(achieved / 1e9, 1), bound="hbm" if hbm_bound else "compute",
                   frac_of_roofline=round(achieved / attainable, 4),
                   n_explore_measured=res.n_explore_measured,
                   n_droplet_measured=res.n_droplet_measured,
                   n_failed=res.n_failed, droplet_moves=res.n_moves,
                   seed_point_us=round(res.seed_ms * 1e3, 3),
                   explore_s=round(res.explore_s, 2), droplet_s=round(res.droplet_s, 2))
        if args.flush:
            row["cold_us"] = round(cold_time(L, task, res.best, stream) * 1e3, 3)
        per_task.append(row)

    # Roofline of the dominant kernel (largest weighted tuned time).
    j = max(range(len(T)), key=lambda i: T[i]["count"] * chosen[i][1].median_ms)
    task, (res, m) = T[j], chosen[j]
    avg_ms = m.mean_ms
    kname = per_task[j]["kernel"]
    if per_task[j]["bound"] == "hbm":
        ach = task["bytes"] / (avg_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                    "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4)}
    else:
        ach = task["flops"] / (avg_ms * 1e-3) / 1e12
        roofline = {"bound": "mfma" if per_task[j]["best_schedule"].get("mfma", 0) else "alu",
                    "achieved": round(ach, 3), "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(ach / PEAK_FP32_TFLOPS, 4)}
    geom = task["space"].geometry(res.best.index())
    roofline.update({"traffic": measured_traffic(kname, per_task[j]["best_schedule"], task["shape"]),
                     "kernel": kname, "task": task["name"],
                     "grid_threads": int(geom["grid"]) * int(geom["threads"]),
                     "avg_launch_us": round(avg_ms * 1e3, 3),
                     "algorithmic_flops": task["flops"], "algorithmic_bytes": task["bytes"]})

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(T, chosen, args.cpu_seconds, L)

    if single:
        cfg_desc = {"workload": describe(T[0]["op"], T[0]["shape"]), "shape": list(T[0]["shape"])}
    else:
        batch = "batch 1" if args.workload == "resnet50" else "batch 16"
        cfg_desc = {"workload": f"{args.workload}: {len(T)} distinct layers ({batch}, fp32)",
                    "layers": [t["name"] for t in T]}
    cfg_desc.update({"n_explore": args.n_explore, "droplet_budget": args.budget})
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
        "data": ("synthetic: SplitMix64 U[-1,1) inputs, seeded" if kind == "uniform" else
                 "synthetic: SplitMix64 N(0,1) inputs and He-normal weights, seeded"),
        "config": cfg_desc,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "tuning": {
            "n_measured_total": sum(r["n_explore_measured"] + r["n_droplet_measured"]
                                    for r in per_task),
            "per_step_gflops": [round(g, 1) for g in gfs],
            "empty_kernel_floor_us": round(floor.median_ms * 1e3, 3),
            "device": info,
        },
    }
    if single:
        r = per_task[0]
        out["tuning"].update({
            "best_schedule": r["best_schedule"], "best_median_us": r["best_us"],
            "n_explore_measured": r["n_explore_measured"],
            "n_droplet_measured": r["n_droplet_measured"], "n_failed": r["n_failed"],
            "droplet_moves": r["droplet_moves"], "seed_point_us": r["seed_point_us"],
            "tuning_wall_s": round(r["explore_s"] + r["droplet_s"], 2),
            "explore_s": r["explore_s"], "droplet_s": r["droplet_s"]})
        if args.flush:
            out["tuning"]["cold_us"] = r["cold_us"]
    else:
        out["tuning"]["network_time_us"] = round(sum(r["count"] * r["best_us"] for r in per_task), 3)
        out["tuning"]["tuning_wall_s"] = round(sum(r["explore_s"] + r["droplet_s"]
                                                   for r in per_task), 2)
        out["tasks"] = per_task
    print(json.dumps(out), flush=True)
    return 0


def cold_time(L, task, best, stream, reps=11, flush_mb=512):
    """Median time (ms) of single launches, each after 512 MB of writes evicted the caches."""
    import torch
    scratch = torch.empty(flush_mb * (1 << 20) // 4, dtype=torch.float32, device="cuda:0")
    times = []
    for _ in range(reps):
        scratch.fill_(1.0)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        L.kernel_run(task["op"], best, task["xd"], task["wd"], task["yd"], stream)
        b.record(stream)
        b.synchronize()
        times.append(a.elapsed_time(b))
    del scratch
    return sorted(times)[reps // 2]


def measured_traffic(kname, knobs, shape):
    """HBM bytes per launch of this kernel instance at this schedule and
    problem shape from the committed rocprofv3 counter runs (FETCH_SIZE and
    WRITE_SIZE, each scaled by the same counter on a copy of known size), or
    None when that schedule was not profiled or the kernel sources changed
    since."""
    from paper_2406_20037_amd.prof_summary import source_hash, traffic_key
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        data = json.load(fh)
    e = data.get(traffic_key(kname, ",".join(f"{k}={v}" for k, v in knobs.items()), shape))
    if not e or e.get("source_sha256") != source_hash(kname):
        return None
    return int(round(e["read_bytes"] + e["write_bytes"]))


def kernel_name(op, knobs, geom):
    """Template instance the schedule selects (as rocprofv3 lists it)."""
    if op == 2:
        if knobs["mfma"]:
            return (f"mm_mfma<{geom['t0']}, {geom['t1']}, {knobs['bk']}, {geom['unroll_eff']}, "
                    f"{knobs['dbuf']}, {geom['threads'] // 256}>")
        return (f"mm_valu<{geom['t0']}, {geom['t1']}, {knobs['bk']}, {geom['unroll_eff']}, "
                f"{knobs['dbuf']}>")
    fam = "conv_mfma" if knobs["mfma"] else "conv_valu"
    return f"{fam}<{geom['t0']}, {geom['t1']}, {geom['unroll_eff']}, {knobs['lds']}>"


def cpu_baseline(T, chosen, min_seconds, L):
    """The fp64 oracle on the host cores over every task of the workload (each
    once per pass), repeated until min_seconds elapse; also the largest
    relative error of the tuned kernels against it."""
    import numpy as np
    import torch

    from oracle import kernels as ok

    threads = ok.num_threads()
    runs, t, flops_done = 0, 0.0, 0
    worst = 0.0
    while runs == 0 or t < min_seconds:
        for task, (res, _) in zip(T, chosen):
            t0 = time.perf_counter()
            ref = (ok.conv2d_f64(task["x"], task["w"], task["shape"]) if task["op"] == 1
                   else ok.matmul_f64(task["x"], task["w"]))
            t += time.perf_counter() - t0
            flops_done += task["flops"]
            if runs == 0:
                L.kernel_run(task["op"], res.best, task["xd"], task["wd"], task["yd"])
                torch.cuda.synchronize()
                y = task["yd"].cpu().numpy().astype(np.float64)
                scale = float(np.abs(ref).max()) or 1.0
                worst = max(worst, float(np.abs(y - ref.ravel()).max()) / scale)
            del ref
        runs += 1
    what = "the full workload" if len(T) == 1 else f"all {len(T)} tasks of the workload"
    return {
        "value": round(flops_done / t / 1e9, 2),
        "unit": "GFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"{what}, {runs} pass(es) in {t:.1f} s (fp64 accumulation, OpenMP)",
        "tuned_kernel_max_rel_err": worst,
    }


if __name__ == "__main__":
    sys.exit(main())
