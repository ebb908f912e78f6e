"""Experiment drivers over the C ABI (no oracle, no CPU fallback): the
exploitation-strategy comparison (Section 3, RQ4; Droplet Search, its variant
with line steps, Random, Grid and GA), the exploration-budget sweep
(RQ5) and the whole-network trial split (Section 2.1).  Each prints one JSON
object per result line on stdout and progress on stderr.

    python -m paper_2406_20037_amd.experiments exploiters --workload matmul_1024 --seeds 3
    python -m paper_2406_20037_amd.experiments exploiters --workload vgg16:L6_256_256_56
    python -m paper_2406_20037_amd.experiments sweep --workload conv3x3_c64_56 --seeds 3
    python -m paper_2406_20037_amd.experiments tasks --workload resnet50 --trials 24,300,1000
    python -m paper_2406_20037_amd.experiments report out/*.jsonl

Every reported kernel time is re-measured with 31 repeats (graph replays) so
that strategies are compared on one footing; tuning-time figures are the
library's own wall-clock of each phase.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

BEST = "best_us"
KIND_NAMES = {0: "droplet", 1: "random", 2: "grid", 3: "ga", 4: "droplet-line"}
CONFIG_OF = {"conv3x3_c64_56": 0, "matmul_1024": 1, "conv7x7_s2_c3_224": 2}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def emit(obj):
    print(json.dumps(obj), flush=True)


class Task:
    """Device inputs and the space of one kernel shape."""

    def __init__(self, L, name, op, shape, kind, stream):
        import torch

        import synthdata
        from synthdata import workloads as wl
        if op == wl.OP_CONV:
            x, w = synthdata.conv_inputs(shape, kind)
            P, Q = synthdata.conv_out_hw(shape[2], shape[3], shape[5], shape[6], shape[7], shape[8])
            n_out = shape[0] * shape[4] * P * Q
        else:
            x, w = synthdata.matmul_inputs(shape, kind)
            n_out = shape[0] * shape[1]
        self.name, self.op, self.shape = name, op, shape
        self.xd, self.wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
        self.yd = torch.empty(n_out, dtype=torch.float32, device="cuda:0")
        self.space = L.Space(op, shape)
        self.io = L.make_io(self.xd, self.wd, self.yd, None, stream)
        self.flops = wl.flops(op, shape)
        self.L = L
        self.final = L.measure_cfg(repeat=31, min_repeat_ms=2.0, max_number=1000, check=0)

    def retime_us(self, sched):
        return self.L.ds_measure(sched, self.io, self.final).median_ms * 1e3


def single_task(L, workload, stream):
    """A single kernel or one layer of a network ("vgg16:L6_256_256_56");
    returns the task and the base seed of its exploration stream."""
    from synthdata import workloads as wl
    if ":" in workload:
        net, layer = workload.split(":", 1)
        layers, config = {"resnet50": (wl.RESNET50, 3), "vgg16": (wl.VGG16, 4)}[net]
        j = next(i for i, (n, _, _, _) in enumerate(layers) if n == layer)
        _, op, shape, _ = layers[j]
        return Task(L, workload, op, shape, "he", stream), wl.sampler_seed(config, j)
    op, shape = wl.SINGLE[workload]
    return Task(L, workload, op, shape, "uniform", stream), wl.sampler_seed(CONFIG_OF[workload])


def run_exploiters(L, args, stream):
    from synthdata import workloads as wl
    task, base_seed = single_task(L, args.workload, stream)
    for s in range(args.seeds):
        seed = base_seed + s
        cache = L.Cache(task.space)
        ex, _ = L.ds_explore(task.space, cache, L.tune_cfg(n_explore=args.n_explore, seed=seed),
                             task.io)
        start = ex.seed_point
        seed_us = task.retime_us(start)
        log(f"seed {seed}: explored {ex.n_explore_measured} in {ex.explore_s:.1f} s, best "
            f"{task.space.knobs(start)} {seed_us:.2f} us")
        for kind in (0, 4, 1, 2, 3):
            for valid_only in ((0,) if kind in (0, 4) else (0, 1)):
                ecfg = L.exploit_cfg(kind=kind, budget=args.budget, seed=seed + 1,
                                     valid_only=valid_only)
                res, _ = L.ds_exploit(task.space, start, ecfg, L.tune_cfg(), task.io,
                                      cache=cache.clone())
                best_us = task.retime_us(res.best)
                row = dict(experiment="exploiters", workload=args.workload, seed=seed,
                           n_explore=ex.n_explore_measured, explore_s=round(ex.explore_s, 3),
                           seed_us=round(seed_us, 3), strategy=KIND_NAMES[kind],
                           valid_only=valid_only, best_us=round(best_us, 3),
                           gflops=round(task.flops / (best_us * 1e-6) / 1e9, 1),
                           speedup_over_seed=round(seed_us / best_us, 4),
                           measured=res.n_droplet_measured, failed=res.n_failed,
                           exploit_s=round(res.droplet_s, 3),
                           best_schedule=task.space.knobs(res.best))
                log(f"  {KIND_NAMES[kind]:8s} valid_only={valid_only}: {best_us:.2f} us, "
                    f"{res.n_droplet_measured} trials ({res.n_failed} failed), {res.droplet_s:.2f} s")
                emit(row)


def run_sweep(L, args, stream):
    from synthdata import workloads as wl
    task, base_seed = single_task(L, args.workload, stream)
    ns = [int(v) for v in args.ns.split(",")]
    for s in range(args.seeds):
        seed = base_seed + s
        for n in ns:
            res, _ = L.ds_tune(task.space, L.tune_cfg(n_explore=n, budget=args.budget, seed=seed),
                               task.io)
            best_us = task.retime_us(res.best)
            row = dict(experiment="sweep", workload=args.workload, seed=seed, n_explore=n,
                       n_explore_measured=res.n_explore_measured,
                       n_droplet_measured=res.n_droplet_measured, moves=res.n_moves,
                       seed_us=round(res.seed_ms * 1e3, 3), best_us=round(best_us, 3),
                       gflops=round(task.flops / (best_us * 1e-6) / 1e9, 1),
                       explore_s=round(res.explore_s, 3), droplet_s=round(res.droplet_s, 3),
                       seed_schedule=task.space.knobs(res.seed_point),
                       best_schedule=task.space.knobs(res.best))
            log(f"seed {seed} N={n}: droplet {res.n_droplet_measured} trials, {best_us:.2f} us, "
                f"{res.wall_s:.1f} s")
            emit(row)
    if args.random_10k:
        cache = L.Cache(task.space)
        seed = base_seed + 999
        ex, _ = L.ds_explore(task.space, cache, L.tune_cfg(n_explore=10000, seed=seed), task.io)
        best_us = task.retime_us(ex.seed_point)
        row = dict(experiment="sweep", workload=args.workload, seed=seed, n_explore=10000,
                   n_explore_measured=ex.n_explore_measured, n_droplet_measured=0,
                   random_only=True, best_us=round(best_us, 3),
                   gflops=round(task.flops / (best_us * 1e-6) / 1e9, 1),
                   explore_s=round(ex.explore_s, 3), best_schedule=task.space.knobs(ex.seed_point))
        log(f"random-10k: {ex.n_explore_measured} points, {best_us:.2f} us, {ex.explore_s:.1f} s")
        emit(row)


def run_tasks(L, args, stream):
    from synthdata import workloads as wl
    if args.workload == "resnet50":
        layers, kind, config = wl.RESNET50, "he", 3
    elif args.workload == "vgg16":
        layers, kind, config = wl.VGG16, "he", 4
    else:
        raise SystemExit("tasks needs a network workload (resnet50 or vgg16)")
    tasks = [Task(L, n, op, sh, kind, stream) for n, op, sh, _ in layers]
    weights = [c for _, _, _, c in layers]
    seeds = [wl.sampler_seed(config, j) for j in range(len(layers))]
    for K in [int(v) for v in args.trials.split(",")]:
        t0 = time.perf_counter()
        results, rounds, net_ms = L.ds_tune_tasks([t.space for t in tasks], weights, seeds, K,
                                                  L.tune_cfg(budget=args.budget),
                                                  ios=[t.io for t in tasks])
        wall = time.perf_counter() - t0
        retimed = [t.retime_us(r.best) for t, r in zip(tasks, results)]
        net_us = sum(w * us for w, us in zip(weights, retimed))
        row = dict(experiment="tasks", workload=args.workload, total_trials=K,
                   quota=rounds[0][1] if rounds else 0, rounds=len(rounds),
                   explore_trials=sum(r.n_explore_measured for r in results),
                   droplet_trials=sum(r.n_droplet_measured for r in results),
                   network_us=round(net_us, 3), network_us_tuning=round(net_ms * 1e3, 3),
                   wall_s=round(wall, 2),
                   per_task=[dict(name=t.name, weight=w, explore=r.n_explore_measured,
                                  droplet=r.n_droplet_measured, best_us=round(us, 3))
                             for t, w, r, us in zip(tasks, weights, results, retimed)])
        log(f"K={K}: network {net_us:.1f} us, explore {row['explore_trials']}, droplet "
            f"{row['droplet_trials']}, {wall:.1f} s")
        emit(row)


def _mean(v):
    return sum(v) / len(v)


def report(paths):
    """Markdown tables over the JSON lines the three experiments print."""
    rows = []
    for p in paths:
        with open(p) as fh:
            rows += [json.loads(line) for line in fh if line.strip()]
    out = []
    ex = [r for r in rows if r["experiment"] == "exploiters"]
    for wl in dict.fromkeys(r["workload"] for r in ex):
        rs = [r for r in ex if r["workload"] == wl]
        seeds = list(dict.fromkeys(r["seed"] for r in rs))
        seed_us = [next(r["seed_us"] for r in rs if r["seed"] == s) for s in seeds]
        out.append(f"{wl}: {len(seeds)} seeds, best of {rs[0]['n_explore']} samples "
                   f"{_mean(seed_us):.2f} us (mean)\n")
        out.append("| strategy | invalid points | best us (mean) | per seed | trials | failed | "
                   "exploit s |")
        out.append("|---|---|---:|---|---|---|---|")
        for strat in dict.fromkeys((r["strategy"], r["valid_only"]) for r in rs):
            g = [r for r in rs if (r["strategy"], r["valid_only"]) == strat]
            out.append(
                f"| {strat[0]} | {'skipped' if strat[1] else 'count'} | "
                f"{_mean([r['best_us'] for r in g]):.2f} | "
                f"{' / '.join(f'{r[BEST]:.2f}' for r in g)} | "
                f"{' / '.join(str(r['measured']) for r in g)} | "
                f"{' / '.join(str(r['failed']) for r in g)} | "
                f"{_mean([r['exploit_s'] for r in g]):.2f} |")
        out.append("")
    sw = [r for r in rows if r["experiment"] == "sweep"]
    for wl in dict.fromkeys(r["workload"] for r in sw):
        rs = [r for r in sw if r["workload"] == wl]
        out.append(f"{wl}: exploration budget N, then Droplet from the best sample\n")
        out.append("| N | best us per seed | mean | Droplet trials per seed | explore s | "
                   "Droplet s |")
        out.append("|---:|---|---:|---|---:|---:|")
        for n in sorted(dict.fromkeys(r["n_explore"] for r in rs)):
            g = [r for r in rs if r["n_explore"] == n]
            name = f"{n} (random only, {g[0]['n_explore_measured']} points)" \
                if g[0].get("random_only") else str(n)
            out.append(
                f"| {name} | {' / '.join(f'{r[BEST]:.2f}' for r in g)} | "
                f"{_mean([r['best_us'] for r in g]):.2f} | "
                f"{' / '.join(str(r['n_droplet_measured']) for r in g)} | "
                f"{_mean([r['explore_s'] for r in g]):.2f} | "
                f"{_mean([r.get('droplet_s', 0.0) for r in g]):.2f} |")
        out.append("")
    ts = [r for r in rows if r["experiment"] == "tasks"]
    for wl in dict.fromkeys(r["workload"] for r in ts):
        rs = [r for r in ts if r["workload"] == wl]
        out.append(f"{wl}: {len(rs[0]['per_task'])} tasks, network time = weighted sum of the "
                   "re-measured per-task best\n")
        out.append("| total exploration trials | first-round quota | rounds | Droplet trials | "
                   "network us | wall s |")
        out.append("|---:|---:|---:|---:|---:|---:|")
        for r in rs:
            out.append(f"| {r['total_trials']} | {r['quota']} | {r['rounds']} | "
                       f"{r['droplet_trials']} | {r['network_us']:.1f} | {r['wall_s']:.1f} |")
        out.append("")
    return "\n".join(out)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("experiment", choices=["exploiters", "sweep", "tasks", "report"])
    ap.add_argument("files", nargs="*", help="report: JSON-lines files the experiments wrote")
    ap.add_argument("--workload", default="matmul_1024")
    ap.add_argument("--seeds", type=int, default=3)
    ap.add_argument("--n-explore", type=int, default=300)
    ap.add_argument("--budget", type=int, default=100)
    ap.add_argument("--ns", default="1,10,25,50,100,200,300,1000")
    ap.add_argument("--random-10k", action="store_true")
    ap.add_argument("--trials", default="24,300,1000,2400")
    args = ap.parse_args(argv)
    if args.experiment == "report":
        print(report(args.files))
        return 0

    import torch

    from paper_2406_20037_amd import _lib as L
    assert torch.cuda.is_available(), "the experiments measure on a GPU"
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    {"exploiters": run_exploiters, "sweep": run_sweep, "tasks": run_tasks}[args.experiment](
        L, args, stream)
    return 0


if __name__ == "__main__":
    sys.exit(main())
