"""Runs one schedule repeatedly (and a plain device copy of known size), for
profiling a single kernel instance with rocprofv3.

    python -m paper_2406_20037_amd.prof_run --workload matmul_1024 \
        --sched bm=64,bn=32,bk=32,unroll=64,dbuf=1,mfma=1,ks=2 --iters 100

The schedule is launched the way the tuner times it: --iters launches captured
in a HIP graph and replayed back to back (--host-launch: one host launch per
iteration instead; with --flush-mb, each after a write of that many MiB that
evicts the caches).  The copy (torch's elementwise copy of --copy-mib MiB)
gives the factor that relates the HBM counters to bytes actually moved.
"""
from __future__ import annotations

import argparse
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="matmul_1024",
                    help="a single-kernel workload, a network layer (resnet50:NAME, vgg16:NAME) "
                         "or a conv shape (conv:N,C,H,W,K,R,S,stride,pad; He-normal inputs)")
    ap.add_argument("--sched", help="knob=value,... (every axis)")
    ap.add_argument("--mfma-ceiling", action="store_true",
                    help="launch the library's pure-MFMA calibration kernel --iters times "
                         "instead of a schedule")
    ap.add_argument("--iters", type=int, default=100)
    ap.add_argument("--copy-mib", type=int, default=64)
    ap.add_argument("--host-launch", action="store_true",
                    help="launch from the host one by one instead of a replayed graph")
    ap.add_argument("--flush-mb", type=int, default=0,
                    help="with --host-launch: write this many MiB of scratch before every "
                         "launch, so each one starts with cold L2 and MALL (their 256 MiB)")
    args = ap.parse_args(argv)

    import torch

    import synthdata
    from synthdata import workloads as wl
    from paper_2406_20037_amd import _lib as L

    if args.mfma_ceiling:
        sink = torch.empty(L.DS_MFMA_CEILING_SINK, device="cuda:0")
        m, flop = L.ds_mfma_ceiling(sink, iters=512,
                                    cfg=L.measure_cfg(warmup=1, repeat=args.iters))
        torch.cuda.synchronize()
        print(f"ran {args.iters + 1} x mfma_ceiling_kernel: median {m.median_ms * 1e3:.1f} us, "
              f"{flop / (m.median_ms * 1e-3) / 1e12:.1f} TFLOP/s", flush=True)
        return 0
    if not args.sched:
        ap.error("--sched is required unless --mfma-ceiling")
    if args.workload.startswith("conv:"):   # any conv shape: conv:N,C,H,W,K,R,S,stride,pad
        op, shape = wl.OP_CONV, tuple(int(v) for v in args.workload[5:].split(","))
        kind = "he"
    elif ":" in args.workload:        # a network layer, e.g. vgg16:L6_256_256_56
        net, layer = args.workload.split(":", 1)
        table = {"resnet50": wl.RESNET50, "vgg16": wl.VGG16}[net]
        op, shape = next((o, sh) for name, o, sh, _ in table if name == layer)
        kind = "he"
    else:
        op, shape = wl.SINGLE[args.workload]
        kind = "uniform"
    knobs = {k: int(v) for k, v in (kv.split("=") for kv in args.sched.split(","))}
    space = L.Space(op, shape)
    s = space.sched_of(**knobs)
    if not space.valid(s.index()):
        ap.error(f"{args.sched} is not a valid point of {args.workload}'s space")
    if op == wl.OP_CONV:
        x, w = synthdata.conv_inputs(shape, kind)
        N, C, H, W, K, R, S, st, pd = shape
        n_out = N * K * ((H + 2 * pd - R) // st + 1) * ((W + 2 * pd - S) // st + 1)
    else:
        x, w = synthdata.matmul_inputs(shape, kind)
        n_out = shape[0] * shape[1]
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    yd = torch.empty(n_out, device="cuda:0")
    if args.flush_mb and not args.host_launch:
        ap.error("--flush-mb needs --host-launch")
    if args.host_launch:
        scratch = (torch.empty(args.flush_mb * (1 << 20) // 4, device="cuda:0")
                   if args.flush_mb else None)
        for _ in range(args.iters):
            if scratch is not None:
                scratch.fill_(1.0)
            L.kernel_run(op, s, xd, wd, yd)
    else:
        # a first and a warm-up launch, then a graph of --iters launches replayed
        # twice (warm-up and timed repeat)
        cfg = L.measure_cfg(warmup=1, repeat=1, min_repeat_ms=1e9, max_number=args.iters,
                            check=0, graph=1)
        m = L.ds_measure(s, L.make_io(xd, wd, yd, None, torch.cuda.current_stream()), cfg)
        if m.status != L.DS_OK:
            raise SystemExit(f"measurement of {args.sched} failed: "
                             f"{L.STATUS_NAMES.get(m.status, m.status)}")
    n = args.copy_mib * (1 << 20) // 4
    a = torch.ones(n, device="cuda:0")
    b = torch.empty_like(a)
    for _ in range(args.iters):
        b.copy_(a)
    torch.cuda.synchronize()
    launches = args.iters if args.host_launch else 2 * args.iters + 2
    print(f"ran {launches} x {space.knobs(s)} and {args.iters} x copy of {args.copy_mib} MiB",
          flush=True)


if __name__ == "__main__":
    sys.exit(main())
