"""Builds ``libdroplet.so`` (the C-ABI library) in-tree for gfx950.

Host-only sources are compiled with g++, HIP sources with hipcc.  The two
kernel-instance sources are compiled several times, each time instantiating
one slice of the template-parameter tuples, so the build runs in parallel.

    python -m paper_2406_20037_amd.build [--jobs N] [--slices S]
"""
from __future__ import annotations

import argparse
import os
import shutil
import subprocess
import sys
import time
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libdroplet.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
ARCH = "gfx950"

HOST_SOURCES = ["space.cpp", "tuner.cpp"]
HIP_SOURCES = ["harness.hip", "kern_reduce.hip"]
SLICED_SOURCES = ["kern_conv.hip", "kern_matmul.hip"]

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++20", "-fPIC",
    # packed fp32 instructions are kept out of every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-I", INCLUDE, "-I", CSRC,
              "-I", os.path.join(ROCM, "include"), "-D__HIP_PLATFORM_AMD__"]


def _hipcc():
    p = shutil.which("hipcc") or os.path.join(ROCM, "bin", "hipcc")
    if not os.path.exists(p):
        raise RuntimeError("hipcc not found; the HIP library cannot be built")
    return p


def _run(cmd):
    t0 = time.time()
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return time.time() - t0, out


def _stale(obj, src, headers):
    if not os.path.exists(obj):
        return True
    t = os.path.getmtime(obj)
    return any(os.path.getmtime(f) > t for f in [src, *headers])


def build(jobs: int | None = None, slices: int | None = None, verbose: bool = False,
          incremental: bool = False) -> str:
    """Compile every source (or, with ``incremental``, only stale objects)."""
    jobs = jobs or max(1, min(16, os.cpu_count() or 1))
    slices = slices or max(2, jobs)
    os.makedirs(BUILD, exist_ok=True)
    hipcc = _hipcc()
    steps = []
    objs = []
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        steps.append(["g++", *HOST_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        steps.append([hipcc, *HIP_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    for src in SLICED_SOURCES:
        for s in range(slices):
            obj = os.path.join(BUILD, f"{src}.s{s}.o")
            steps.append([hipcc, *HIP_FLAGS, f"-DDS_SLICE={s}", f"-DDS_NSLICES={slices}", "-c",
                          os.path.join(CSRC, src), "-o", obj])
            objs.append(obj)
    headers = [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".h")]
    headers.append(os.path.join(INCLUDE, "droplet.h"))
    if incremental:
        steps = [c for c in steps if _stale(c[c.index("-o") + 1], c[c.index("-c") + 1], headers)]
    t0 = time.time()
    # the slowest (sliced kernel) steps first
    order = sorted(range(len(steps)), key=lambda i: 0 if "-DDS_SLICE" in " ".join(steps[i]) else 1)
    with ThreadPoolExecutor(jobs) as ex:
        for (dt, out) in ex.map(lambda i: _run(steps[i]), order):
            if verbose and out.strip():
                print(out)
    tmp = LIB + ".tmp"
    _run([hipcc, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB} in {time.time() - t0:.1f}s ({len(steps)} objects, {slices} slices)")
    return LIB


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=None)
    ap.add_argument("--slices", type=int, default=None)
    ap.add_argument("--incremental", action="store_true")
    args = ap.parse_args(argv)
    build(args.jobs, args.slices, verbose=True, incremental=args.incremental)


if __name__ == "__main__":
    sys.exit(main())
