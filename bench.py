"""Benchmark of the tuning hot path on one MI355X.

Set-up (untimed): every task of the five workloads is tuned once by the
combined approach -- 300 exploration samples, then Droplet Search with at
most 100 trials from the best of them -- each task with its own sampler seed:

    conv 3x3 C64 K64 56x56 (batch 1), matmul 1024^3, conv 7x7/2 C3 K64 224x224,
    ResNet-50 at batch 1 (23 distinct conv layers + FC), VGG-16 at batch 16
    (13 conv layers, each tuned independently).

Timed region: one step is one pass of the tuned VGG-16 b16 network -- its 13
conv layers, each launched once in layer order on one stream, inputs resident
in HBM.  `value` is the network's GFLOP/s (491.1 GFLOP per pass over the
event-timed pass time), `ms_per_step` the pass time.  Events between the
layers give each layer's average launch duration inside the same timed
passes; the dominant layer carries the `roofline` object.  The other four
workloads are timed the same way after the headline (a pass = every tuned
kernel of the workload, each as often as the network runs it) and reported
in `configs`, with their tuning counts and wall-clock.

The CPU baseline leg runs the fp64 oracle once over every task of the five
workloads on the host cores, and checks every tuned kernel's output against
it (max |y - ref| <= 1e-4 max |ref|); a failed check makes the run exit 3.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5]
    python bench.py --workloads conv3x3_c64_56,matmul_1024 --no-cpu-baseline
    python bench.py --workloads vgg16 --layers 0-6 --steps 5 --warmup 1
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
TOL = 1e-4

# (workload, config number) in the order the configurations are listed
WORKLOADS = [("conv3x3_c64_56", 0), ("matmul_1024", 1), ("conv7x7_s2_c3_224", 2),
             ("resnet50", 3), ("vgg16", 4)]
HEADLINE = "vgg16"
DESCRIPTION = {
    "conv3x3_c64_56": "conv2d NCHW fp32 N=1 C=64 H=W=56 K=64 3x3 stride 1 pad 1",
    "matmul_1024": "matmul fp32 row-major M=N=K=1024",
    "conv7x7_s2_c3_224": "conv2d NCHW fp32 N=1 C=3 H=W=224 K=64 7x7 stride 2 pad 3",
    "resnet50": "ResNet-50 (v1.5) batch 1 fp32: 23 distinct conv layers + FC 2048x1000",
    "vgg16": "VGG-16 batch 16 fp32: 13 conv layers 3x3 stride 1 pad 1, NCHW",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse_layers(spec, n):
    if not spec:
        return list(range(n))
    idx = []
    for part in spec.split(","):
        a, _, b = part.partition("-")
        idx += list(range(int(a), int(b or a) + 1))
    return idx


def workload_tasks(name, layers=""):
    """[(task name, op, shape, count, layer index)] and the input kind."""
    from synthdata import workloads as wl
    if name in wl.SINGLE:
        op, shape = wl.SINGLE[name]
        return [(name, op, shape, 1, 0)], "uniform"
    tasks = {"resnet50": wl.RESNET50, "vgg16": wl.VGG16}.get(name)
    if tasks is None:
        raise SystemExit(f"unknown workload {name}")
    return [(tasks[i][0], tasks[i][1], tasks[i][2], tasks[i][3], i)
            for i in parse_layers(layers, len(tasks))], "he"


FAMILY_NAME = {1: "conv_valu", 2: "conv_mfma", 3: "mm_valu", 4: "mm_mfma", 5: "conv_mfma2"}


def kernel_name(space, idx):
    """Template instance the schedule selects (as rocprofv3 lists it)."""
    info = space.kernel_info(idx)
    args = ", ".join(str(v) for v in info["params"][: info["nparams"]])
    return f"{FAMILY_NAME[info['family']]}<{args}>"


def roof(flops, nbytes, seconds):
    """(achieved flop/s, attainable, bound) of one kernel launch."""
    ai = flops / nbytes
    hbm_bound = ai * PEAK_HBM_GBS * 1e9 < PEAK_FP32_TFLOPS * 1e12
    attainable = ai * PEAK_HBM_GBS * 1e9 if hbm_bound else PEAK_FP32_TFLOPS * 1e12
    return flops / seconds, attainable, "hbm" if hbm_bound else "compute"


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


def cold_time(L, task, stream, reps=11, flush_mb=512):
    """Median time (ms) of single launches, each after 512 MB of writes evicted the caches."""
    import torch
    scratch = torch.empty(flush_mb * (1 << 20) // 4, dtype=torch.float32, device="cuda:0")
    times = []
    for _ in range(reps):
        scratch.fill_(1.0)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        L.kernel_run(task["op"], task["best"], task["xd"], task["wd"], task["yd"], stream)
        b.record(stream)
        b.synchronize()
        times.append(a.elapsed_time(b))
    del scratch
    return sorted(times)[reps // 2]


class Workload:
    def __init__(self, name, config, layers, L, wl, synthdata, torch):
        self.name, self.config = name, config
        tasks, self.kind = workload_tasks(name, layers)
        self.T = []
        for tname, op, shape, count, layer in tasks:
            if op == wl.OP_CONV:
                x, w = synthdata.conv_inputs(shape, self.kind)
                P, Q = synthdata.conv_out_hw(shape[2], shape[3], shape[5], shape[6], shape[7],
                                             shape[8])
                n_out = shape[0] * shape[4] * P * Q
            else:
                x, w = synthdata.matmul_inputs(shape, self.kind)
                n_out = shape[0] * shape[1]
            xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
            yd = torch.empty(n_out, dtype=torch.float32, device="cuda:0")
            self.T.append(dict(name=tname, op=op, shape=shape, count=count, layer=layer, x=x, w=w,
                               xd=xd, wd=wd, yd=yd, space=L.Space(op, shape),
                               flops=wl.flops(op, shape), bytes=wl.algorithmic_bytes(op, shape)))
        self.flops = sum(t["count"] * t["flops"] for t in self.T)

    def tune(self, L, wl, args, stream, final_cfg):
        t0 = time.perf_counter()
        for task in self.T:
            seed = wl.sampler_seed(self.config, task["layer"])
            cfg = L.tune_cfg(n_explore=args.n_explore, budget=args.budget, seed=seed)
            io = L.make_io(task["xd"], task["wd"], task["yd"], None, stream)
            res, _ = L.ds_tune(task["space"], cfg, io)
            m = L.ds_measure(res.best, io, final_cfg)
            task.update(best=res.best, res=res, meas=m,
                        knobs=task["space"].knobs(res.best),
                        geom=task["space"].geometry(res.best.index()))
            task["kernel"] = kernel_name(task["space"], res.best.index())
            log(f"tuned {self.name}/{task['name']}: {task['knobs']} {m.median_ms * 1e3:.2f} us "
                f"({task['flops'] / (m.median_ms * 1e-3) / 1e9:.0f} GFLOP/s), explored "
                f"{res.n_explore_measured}, droplet {res.n_droplet_measured}, "
                f"{res.explore_s + res.droplet_s:.2f} s")
        self.tune_wall = time.perf_counter() - t0

    def one_pass(self, L, stream, evs=None):
        """Every task launched `count` times, in order, on `stream`; evs[i+1]
        is recorded after task i when given."""
        for i, task in enumerate(self.T):
            for _ in range(task["count"]):
                L.kernel_run(task["op"], task["best"], task["xd"], task["wd"], task["yd"], stream)
            if evs is not None:
                evs[i + 1].record(stream)

    def timed_passes(self, L, torch, stream, warmup, steps):
        """Host-launched passes timed with events on `stream` after `warmup`
        untimed ones; returns (ms per pass, per-task mean ms per launch inside
        the timed passes)."""
        for _ in range(warmup):
            self.one_pass(L, stream)
        torch.cuda.synchronize()
        all_evs = []
        for _ in range(steps):
            evs = [torch.cuda.Event(enable_timing=True) for _ in range(len(self.T) + 1)]
            evs[0].record(stream)
            self.one_pass(L, stream, evs)
            all_evs.append(evs)
        torch.cuda.synchronize()
        total = all_evs[0][0].elapsed_time(all_evs[-1][-1])
        launch_ms = [sum(e[i].elapsed_time(e[i + 1]) for e in all_evs) / (steps * task["count"])
                     for i, task in enumerate(self.T)]
        return total / steps, launch_ms

    def graph_passes(self, L, torch, warmup, steps):
        """Passes captured into one HIP graph (as many back to back as make
        it last about 2 ms, from the tuned times) and replayed `steps` times
        between two events (small kernels: host launches would time the
        launch path, and one graph per pass the graph launch).  Returns ms
        per pass."""
        est_ms = sum(t["count"] * t["meas"].median_ms for t in self.T)
        per_graph = max(1, min(1000, int(2.0 / max(est_ms, 1e-4))))
        side = torch.cuda.Stream()
        torch.cuda.synchronize()
        self.one_pass(L, side)            # creates this stream's split workspaces
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            for _ in range(per_graph):
                self.one_pass(L, side)
        for _ in range(warmup):
            g.replay()
        torch.cuda.synchronize()
        cur = torch.cuda.current_stream()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(cur)
        for _ in range(steps):
            g.replay()
        b.record(cur)
        torch.cuda.synchronize()
        del g
        return a.elapsed_time(b) / (steps * per_graph)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workloads", default=",".join(w for w, _ in WORKLOADS),
                    help="comma list of " + ", ".join(w for w, _ in WORKLOADS))
    ap.add_argument("--layers", default="", help="network workloads: task indices, e.g. 0-6,9")
    ap.add_argument("--n-explore", type=int, default=300)
    ap.add_argument("--budget", type=int, default=100)
    ap.add_argument("--flush", action="store_true",
                    help="also time each tuned kernel cold (512 MB written between launches)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}): the tuner and the timed "
              "passes run on a single device; there is no multi-GPU mode.", file=sys.stderr)
        return 2

    import torch

    import synthdata
    from synthdata import workloads as wl
    from paper_2406_20037_amd import _lib as L

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    info = L.ds_device_info()
    names = [w for w in args.workloads.split(",") if w]
    cfg_of = dict(WORKLOADS)
    for n in names:
        if n not in cfg_of:
            raise SystemExit(f"unknown workload {n}")
    head = HEADLINE if HEADLINE in names else names[-1]
    log(f"device {info}; workloads {names}; headline {head}")

    # Inputs of every task, resident on the device before any tuning or timing.
    W = {n: Workload(n, cfg_of[n], args.layers if n in ("resnet50", "vgg16") else "", L, wl,
                     synthdata, torch) for n in names}

    # Set-up: tune every task once (300 samples + Droplet <= 100).
    final_cfg = L.measure_cfg(repeat=31, min_repeat_ms=2.0, max_number=1000, check=0)
    for n in names:
        W[n].tune(L, wl, args, stream, final_cfg)
    floor = L.ds_empty_kernel_floor(stream)
    # The fp32 MFMA rate this device sustains with no memory traffic (the
    # library's calibration launch), beside the published peak.
    sink = torch.empty(L.DS_MFMA_CEILING_SINK, device="cuda:0")
    ceil_m, ceil_flop = L.ds_mfma_ceiling(sink, iters=512, stream=stream,
                                          cfg=L.measure_cfg(repeat=7))
    ceiling_tflops = ceil_flop / (ceil_m.median_ms * 1e-3) / 1e12
    del sink

    # Timed region: passes of the headline network, then of the other workloads.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ms_step, launch_ms = W[head].timed_passes(L, torch, stream, args.warmup, args.steps)
    wall = time.perf_counter() - t0
    value = W[head].flops / (ms_step * 1e-3) / 1e9
    log(f"{head}: {ms_step:.3f} ms per pass, {value:.1f} GFLOP/s (wall {wall:.2f} s)")
    pass_ms = {head: ms_step}
    for n in names:
        if n != head:
            pass_ms[n] = W[n].graph_passes(L, torch, max(args.warmup, 3), max(args.steps, 20))
            log(f"{n}: {pass_ms[n] * 1e3:.2f} us per pass "
                f"({W[n].flops / (pass_ms[n] * 1e-3) / 1e9:.1f} GFLOP/s)")

    # CPU baseline leg: the oracle on the host cores, and the oracle check
    # of every tuned kernel (outside the timed region).
    cpu, worst = None, None
    if not args.no_cpu_baseline:
        cpu, worst = cpu_baseline(W, names, L, torch, stream)

    # Per-workload rows (configs) and per-task rows.
    configs = []
    for n in names:
        wk = W[n]
        rows = []
        for i, task in enumerate(wk.T):
            res, m = task["res"], task["meas"]
            ach, att, bound = roof(task["flops"], task["bytes"], m.median_ms * 1e-3)
            rows.append(dict(
                name=task["name"], count=task["count"], shape=list(task["shape"]),
                best_schedule=task["knobs"], kernel=task["kernel"],
                tuned_us=round(m.median_ms * 1e3, 3),
                gflops=round(ach / 1e9, 1), bound=bound, frac_of_roofline=round(ach / att, 4),
                n_explore_measured=res.n_explore_measured,
                n_droplet_measured=res.n_droplet_measured, n_failed=res.n_failed,
                droplet_moves=res.n_moves, seed_point_us=round(res.seed_ms * 1e3, 3),
                tuning_wall_s=round(res.explore_s + res.droplet_s, 2),
                max_rel_err=task.get("max_rel_err")))
            if n == head:
                rows[-1]["launch_us"] = round(launch_ms[i] * 1e3, 3)
            if args.flush:
                rows[-1]["cold_us"] = round(cold_time(L, task, stream) * 1e3, 3)
        dom = max(range(len(rows)), key=lambda i: rows[i]["count"] * rows[i]["tuned_us"])
        pm = pass_ms[n]
        configs.append(dict(
            config=wk.config, workload=DESCRIPTION[n], name=n,
            gflops=round(wk.flops / (pm * 1e-3) / 1e9, 1),
            frac_of_fp32_peak=round(wk.flops / (pm * 1e-3) / (PEAK_FP32_TFLOPS * 1e12), 4),
            pass_us=round(pm * 1e3, 3),
            pass_timing=("host launches, events" if n == head else
                         "graph replays (passes back to back in one graph), events"),
            dominant_task=rows[dom]["name"],
            dominant_frac_of_roofline=rows[dom]["frac_of_roofline"],
            n_explore_measured=sum(r["n_explore_measured"] for r in rows),
            n_droplet_measured=sum(r["n_droplet_measured"] for r in rows),
            tuning_wall_s=round(wk.tune_wall, 2),
            tasks=rows))

    # Roofline of the headline's dominant kernel, from the timed passes.
    hc = next(c for c in configs if c["name"] == head)
    j = max(range(len(W[head].T)), key=lambda i: W[head].T[i]["count"] * launch_ms[i])
    task = W[head].T[j]
    avg_ms = launch_ms[j]
    ach, att, bound = roof(task["flops"], task["bytes"], avg_ms * 1e-3)
    if bound == "hbm":
        roofline = {"bound": "hbm", "achieved": round(task["bytes"] / (avg_ms * 1e-3) / 1e9, 1),
                    "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    else:
        roofline = {"bound": "mfma" if task["knobs"].get("mfma", 0) else "alu",
                    "achieved": round(ach / 1e12, 3), "peak": PEAK_FP32_TFLOPS,
                    "unit": "TFLOP/s"}
    roofline["frac"] = round(roofline["achieved"] / roofline["peak"], 4)
    if roofline["unit"] == "TFLOP/s":
        roofline["mfma_ceiling"] = round(ceiling_tflops, 2)
        roofline["frac_of_ceiling"] = round(roofline["achieved"] / ceiling_tflops, 4)
    # A split schedule is two launches per layer (the kernel, then the reduce
    # of its partial outputs): the events time both, and so does the traffic.
    splits = task["space"].kernel_info(task["best"].index())["splits"]
    traffic = measured_traffic(task["kernel"], task["knobs"], task["shape"])
    if splits > 1:
        red = f"split_reduce_kernel<{splits}>"
        n4 = -(-int(task["yd"].numel()) // 4)          # the reduce's launch: float4 lanes,
        roofline.update({"reduce_kernel": red,         # 256-thread blocks, at most 4096
                         "reduce_grid_threads": min(-(-n4 // 256), 4096) * 256})
        rt = measured_traffic(red, task["knobs"], task["shape"])
        traffic = traffic + rt if traffic is not None and rt is not None else None
    roofline.update({"traffic": traffic,
                     "kernel": task["kernel"], "task": task["name"],
                     "schedule": task["knobs"],
                     "grid_threads": int(task["geom"]["grid"]) * int(task["geom"]["threads"]),
                     "avg_launch_us": round(avg_ms * 1e3, 3),
                     "algorithmic_flops": task["flops"], "algorithmic_bytes": task["bytes"]})

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic, seeded (SplitMix64): U[-1,1) inputs for the single kernels; "
                "N(0,1) inputs and He-normal weights for ResNet-50 and VGG-16",
        "config": {"workload": DESCRIPTION[head] + (f" (layers {args.layers})" if args.layers
                                                    and head in ("resnet50", "vgg16") else ""),
                   "step": "one pass of the tuned network: every layer launched once, in order",
                   "layers": [t["name"] for t in W[head].T],
                   "n_explore": args.n_explore, "droplet_budget": args.budget},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "configs": configs,
        "tuning": {
            "n_measured_total": sum(c["n_explore_measured"] + c["n_droplet_measured"]
                                    for c in configs),
            "tuning_wall_s_total": round(sum(c["tuning_wall_s"] for c in configs), 2),
            "empty_kernel_floor_us": round(floor.median_ms * 1e3, 3),
            "mfma_ceiling_tflops": round(ceiling_tflops, 2),
            "device": info,
        },
        "parity": None if worst is None else {
            "tolerance": TOL, "max_rel_err": worst,
            "status": "ok" if worst <= TOL else "FAIL"},
    }
    print(json.dumps(out), flush=True)
    if worst is not None and not worst <= TOL:
        log(f"a tuned kernel fails the oracle check: max relative error {worst:.3g} > {TOL}")
        return 3
    return 0


def cpu_baseline(W, names, L, torch, stream):
    """The fp64 oracle (C, OpenMP) on the host cores: every task of every
    workload once, timed; each tuned kernel's output is checked against it."""
    import numpy as np

    from oracle import kernels as ok

    threads = ok.num_threads()
    t, flops_done, n_tasks = 0.0, 0, 0
    worst = 0.0
    for n in names:
        wk = W[n]
        for task in wk.T:
            sh = task["shape"]
            t0 = time.perf_counter()
            if task["op"] == 1:
                ref = ok.conv2d_f64(task["x"], task["w"], sh)
            else:
                ref = ok.matmul_f64(task["x"], task["w"])
            t += time.perf_counter() - t0
            flops_done += task["flops"]
            n_tasks += 1
            task["yd"].fill_(float("nan"))
            L.kernel_run(task["op"], task["best"], task["xd"], task["wd"], task["yd"], stream)
            torch.cuda.synchronize()
            y = task["yd"].cpu().numpy().astype(np.float64)
            ref = ref.ravel()
            scale = float(np.abs(ref).max()) or 1.0
            err = float(np.abs(y - ref).max()) / scale if np.all(np.isfinite(y)) else float("inf")
            task["max_rel_err"] = err
            worst = max(worst, err)
            log(f"oracle check {n}/{task['name']}: max rel err {err:.3g}")
            del ref, y
    return {
        "value": round(flops_done / t / 1e9, 2),
        "unit": "GFLOP/s",
        "cores": threads,
        "affinity_cpus": len(os.sched_getaffinity(0)),
        "kind": "oracle",
        "sample": f"every task of {', '.join(names)} once ({n_tasks} kernels, "
                  f"{flops_done / 1e9:.1f} GFLOP of fp64-accumulated work) in {t:.1f} s; "
                  f"OpenMP threads {threads}",
        "tuned_kernel_max_rel_err": worst,
    }, worst


if __name__ == "__main__":
    sys.exit(main())
