"""Summarises rocprofv3 SQLite outputs (kernel-trace stats and --pmc runs) as
Markdown tables.

    python -m paper_2406_20037_amd.prof_summary --trace RUN_results.db \
        [--fetch FETCH_results.db --write WRITE_results.db --copy-mib 64] [--top 15]

FETCH_SIZE / WRITE_SIZE are KiB per dispatch; each is scaled by the ratio of
the known byte count of the plain copy kernel (``__amd_rocclr_copyBuffer`` of
--copy-mib MiB) to what the same counter reads for it.
"""
from __future__ import annotations

import argparse
import collections
import hashlib
import json
import os
import re
import sqlite3
import sys

COPY = "__amd_rocclr_copyBuffer"
PKG = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCES = {
    "mm_": ["csrc/kern_matmul.hip", "csrc/kern_common.h", "csrc/ds_internal.h"],
    "conv_": ["csrc/kern_conv.hip", "csrc/kern_common.h", "csrc/ds_internal.h"],
    "split_reduce_kernel": ["csrc/kern_reduce.hip", "csrc/kern_reduce.h", "csrc/kern_common.h"],
}


_COMMENT = re.compile(r"/\*.*?\*/|//[^\n]*", re.S)


def code_digest(paths) -> str:
    """sha256 over the code of the given source files: comments removed and
    whitespace runs collapsed, so an edit to a comment keeps the digest."""
    h = hashlib.sha256()
    for p in paths:
        with open(p, encoding="utf-8") as fh:
            text = _COMMENT.sub(" ", fh.read())
        h.update(" ".join(text.split()).encode())
        h.update(b"\0")
    return h.hexdigest()


def source_hash(kernel: str) -> str | None:
    """Code digest of the source files a kernel family is compiled from."""
    for prefix, files in KERNEL_SOURCES.items():
        if kernel.startswith(prefix):
            return code_digest(os.path.join(PKG, f) for f in files)
    return None


# Position of the unroll-factor template argument of each kernel family.
UNROLL_ARG = {"mm_mfma": 3, "mm_valu": 3, "conv_mfma": 2, "conv_valu": 2, "conv_mfma2": 2}


def traffic_key(kernel: str, sched: str, shape=None) -> str:
    """Key of a kernel's HBM traffic entry: the instance and the schedule (the
    same instance runs with different runtime tile arguments).  The unroll knob
    and the instance's unroll factor are left out: they order instructions and
    set how far ahead operands are read, but never change the addresses a
    launch reads or writes.  Band tiles (conv mfma 3) are th * tw consecutive
    output pixels, so their th and tw enter only as that product (npx).  The
    problem shape, when given, ends the key."""
    name = kernel
    if "<" in kernel and kernel.endswith(">"):
        fam, args = kernel[:-1].split("<", 1)
        parts = [a.strip() for a in args.split(",")]
        pos = UNROLL_ARG.get(fam.strip())
        if pos is not None and pos < len(parts):
            parts[pos] = "*"
        name = f"{fam}<{', '.join(parts)}>"
    kept = [kv for kv in sched.split(",") if kv and not kv.startswith("unroll=")]
    kv = dict(k.split("=", 1) for k in kept)
    if kv.get("mfma") == "3" and "th" in kv and "tw" in kv:
        npx = int(kv["th"]) * int(kv["tw"])
        kept = [k for k in kept if not k.startswith(("th=", "tw="))]
        kept.insert(1 if kept and kept[0].startswith("tk=") else 0, f"npx={npx}")
    key = f"{name} {','.join(kept)}" if kept else name
    if shape:
        key += " shape=" + ",".join(str(int(v)) for v in shape)
    return key


def short(name: str) -> str:
    return (name.replace("ds::(anonymous namespace)::", "").replace("void ", "")
            .replace("(ds::MatmulArgs)", "").replace("(ds::ConvArgs)", "")
            .replace("(ds::Conv2Args)", "").replace("(float const*, float*, long)", ""))


def top_kernels(db, top):
    """Rows of rocprofv3's top_kernels view (durations in microseconds)."""
    cur = sqlite3.connect(db).cursor()
    rows = list(cur.execute("select name, total_calls, total_duration, average, percentage "
                            "from top_kernels"))
    return rows[:top], len(rows)


def counters(db):
    cur = sqlite3.connect(db).cursor()
    acc = collections.defaultdict(list)
    for name, counter, value in cur.execute(
            "select kernel_name, counter_name, value from counters_collection"):
        acc[(name, counter)].append(float(value))
    return {k: sum(v) / len(v) for k, v in acc.items()}, {k: len(v) for k, v in acc.items()}


def paired_reduce(cur, kname, threads, red):
    """(kernel, reduce) duration pairs of the dispatches of kname at the given
    grid that are directly followed (in start time) by a dispatch of red: the
    launches of that split schedule, not the same kernel instance or reduce of
    another task that shares the grid.  Empty when the trace has no start
    times."""
    cols = [c[0] for c in cur.execute("select * from kernels limit 1").description]
    if "start" not in cols:
        return []
    seq = list(cur.execute('select name, start, duration, grid_x * grid_y * grid_z from kernels '
                           'order by start'))
    out = []
    for (name, _, d, g), nxt in zip(seq, seq[1:]):
        if short(name) == kname and (threads is None or g == threads) and short(nxt[0]) == red:
            out.append((d, nxt[2]))
    return out


def bench_check(db, bench_json):
    """The dominant kernel of a profiled bench.py run: its traced dispatches at
    the tuned launch shape against the average launch time bench.py reported
    (HIP events over back-to-back graph launches, so it also holds the gap
    between consecutive kernels)."""
    with open(bench_json) as fh:
        line = [ln for ln in fh if ln.lstrip().startswith("{")][-1]
    rf = json.loads(line)["roofline"]
    kname, threads = rf["kernel"], rf.get("grid_threads")
    red, rgrid = rf.get("reduce_kernel"), rf.get("reduce_grid_threads")
    cur = sqlite3.connect(db).cursor()
    rows = list(cur.execute("select name, duration, grid_x * grid_y * grid_z from kernels"))
    durs = [(d, g) for name, d, g in rows if short(name) == kname]
    pairs = paired_reduce(cur, kname, threads, red) if red else []
    if pairs:
        # a split schedule: its own launches are the ones its reduce follows
        at = sorted(d for d, _ in pairs)
        what_k = "this instance, this grid, followed by the reduce"
    else:
        at = sorted(d for d, g in durs if threads is None or g == threads)
        what_k = "this instance, this grid"
    print(f"\n### Dominant kernel of the profiled bench.py run\n")
    what = f"`{kname}`" + (f" followed by `{red}`" if red else "")
    print(f"bench.py: {what} on task {rf['task']}, average launch {rf['avg_launch_us']:.3f} us "
          f"(events around its launches in the timed passes), {rf['achieved']} {rf['unit']} "
          f"= {rf['frac']:.3f} of {rf['peak']}.\n")
    if not at:
        print("No traced dispatch of that kernel at that launch shape.")
        return
    mean = sum(at) / len(at) / 1e3
    med = at[len(at) // 2] / 1e3
    print(f"| kernel | dispatches ({what_k}) | mean us | median us | min us |")
    print("|---|---:|---:|---:|---:|")
    print(f"| `{kname}` | {len(at)} of {len(durs)} | {mean:.3f} | {med:.3f} | {at[0] / 1e3:.3f} |")
    total = med
    if red:
        rd, how = sorted(r for _, r in pairs), "after each of them"
        if not rd:
            # no dispatch times in the trace: every reduce of that grid
            rd = sorted(d for name, d, g in rows if short(name) == red and (rgrid is None or g == rgrid))
            how = "every dispatch of that grid"
        if rd:
            rmed = rd[len(rd) // 2] / 1e3
            total += rmed
            print(f"| `{red}` ({how}) | {len(rd)} | {sum(rd) / len(rd) / 1e3:.3f} | {rmed:.3f} | "
                  f"{rd[0] / 1e3:.3f} |")
    print(f"\nTraced median per layer launch {total:.3f} us against the bench's "
          f"{rf['avg_launch_us']:.3f} us (difference {rf['avg_launch_us'] - total:.3f} us, "
          f"{(rf['avg_launch_us'] - total) / total * 100:+.1f}%).")


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace", required=True)
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-mib", type=int, default=64)
    ap.add_argument("--top", type=int, default=15)
    ap.add_argument("--counters", nargs="*", default=[],
                    help="further --pmc runs: every counter per kernel (mean per dispatch)")
    ap.add_argument("--json-out", help="merge the scaled HBM bytes of our kernels into this file")
    ap.add_argument("--command", default="", help="recorded with the --json-out entries")
    ap.add_argument("--sched", default="",
                    help="schedule the profiled launches ran (knob=value,... in axis order); "
                         "--json-out entries are keyed by kernel and schedule")
    ap.add_argument("--shape", default="",
                    help="problem shape of the profiled launches (comma-separated); ends the keys")
    ap.add_argument("--bench-json",
                    help="bench.py output of the profiled run: compare its dominant kernel's "
                         "average launch time with the traced dispatch durations")
    args = ap.parse_args(argv)
    rows, n = top_kernels(args.trace, args.top)
    print(f"### Kernel trace ({n} distinct kernels; top {len(rows)} by total time)\n")
    print("| kernel | calls | total us | avg us | % |")
    print("|---|---:|---:|---:|---:|")
    for name, calls, tot, avg, pct in rows:
        print(f"| `{short(name)}` | {calls} | {tot:.1f} | {avg:.3f} | {pct:.1f} |")
    if args.bench_json:
        bench_check(args.trace, args.bench_json)
    if args.fetch and args.write:
        copy_bytes_kib = args.copy_mib * 1024.0
        f, fn = counters(args.fetch)
        w, wn = counters(args.write)
        fc = f.get((COPY, "FETCH_SIZE"))
        wc = w.get((COPY, "WRITE_SIZE"))
        ff = copy_bytes_kib / fc if fc else float("nan")
        wf = copy_bytes_kib / wc if wc else float("nan")
        print(f"\n### HBM counters (KiB per dispatch)\n")
        print(f"Copy kernel of {args.copy_mib} MiB: FETCH_SIZE {fc:.1f} KiB -> read factor "
              f"{ff:.3f}; WRITE_SIZE {wc:.1f} KiB -> write factor {wf:.3f}.\n")
        print("| kernel | dispatches | FETCH_SIZE | WRITE_SIZE | read bytes (scaled) | "
              "write bytes (scaled) |")
        print("|---|---:|---:|---:|---:|---:|")
        names = sorted({k[0] for k in f} | {k[0] for k in w})
        entries = {}
        for name in names:
            fv = f.get((name, "FETCH_SIZE"), float("nan"))
            wv = w.get((name, "WRITE_SIZE"), float("nan"))
            print(f"| `{short(name)}` | {fn.get((name, 'FETCH_SIZE'), 0)} | {fv:.1f} | {wv:.1f} | "
                  f"{fv * ff * 1024:.0f} | {wv * wf * 1024:.0f} |")
            k = short(name)
            sh = source_hash(k)
            if sh:
                shape = [int(v) for v in args.shape.split(",")] if args.shape else None
                entries[traffic_key(k, args.sched, shape)] = {"fetch_kib": fv, "write_kib": wv, "read_factor": ff,
                              "write_factor": wf, "read_bytes": fv * ff * 1024,
                              "write_bytes": wv * wf * 1024, "source_sha256": sh,
                              "command": args.command}
        if args.json_out and entries:
            data = {}
            if os.path.exists(args.json_out):
                with open(args.json_out) as fh:
                    data = json.load(fh)
            data.update(entries)
            with open(args.json_out, "w") as fh:
                json.dump(data, fh, indent=1, sort_keys=True)
    for db in args.counters:
        c, cn = counters(db)
        names = sorted({k[1] for k in c})
        print(f"\n### Counters ({', '.join(names)}; mean per dispatch)\n")
        print("| kernel | dispatches | " + " | ".join(names) + " |")
        print("|---|---:|" + "---:|" * len(names))
        for k in sorted({k[0] for k in c}):
            vals = " | ".join(f"{c.get((k, n), float('nan')):.4g}" for n in names)
            print(f"| `{short(k)}` | {cn.get((k, names[0]), 0)} | {vals} |")
    return 0


if __name__ == "__main__":
    sys.exit(main())
