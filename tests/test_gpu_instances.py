"""Every compiled program the five workloads' lattices can select, on the GPU.

1. Reachable instances.  For every task of the five workloads (conv 3x3 C64
   56x56, matmul 1024^3, conv 7x7/2 C3 224x224, the ResNet-50 layers and FC,
   the VGG-16 layers) the library lists the template instance each valid
   lattice point selects (Definition 1: an annotated sketch is a concrete
   program).  Each distinct instance is launched once, at the first point (in
   key order) of the smallest workload that reaches it, on small-integer
   inputs: every fp32 summation order is then exact, so sampled outputs must
   equal the oracle's fp64 sums bit for bit, every output must be written
   (NaN prefill) and nothing past the output (canary tail).

2. The validity predicate against the compiled code.  For the same instances,
   hipFuncGetAttributes must show no register spill (scratch 0), a launch bound
   that admits the geometry's workgroup, and static + dynamic LDS within the
   163840 bytes a workgroup may use.

3. Tuned winners.  Each task of the five workloads is tuned with a small budget
   and its winner compared with the oracle on every output.
"""
import collections

import numpy as np
import pytest

import synthdata
from synthdata import workloads as wl
from oracle import kernels as ok

pytestmark = pytest.mark.gpu

LDS_LIMIT = 163840
CANARY = 12345.0
TAIL = 64
FAMILY = {1: "conv_valu", 2: "conv_mfma", 3: "mm_valu", 4: "mm_mfma", 5: "conv_mfma2"}


@pytest.fixture(scope="module")
def env():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a device"
    from paper_2406_20037_amd import _lib
    return torch, _lib


def all_tasks():
    out = [(n, op, sh) for n, (op, sh) in wl.SINGLE.items()]
    out += [(n, op, sh) for n, op, sh, _ in wl.RESNET50]
    out += [("vgg_" + n, op, sh) for n, op, sh, _ in wl.VGG16]
    return out


def out_elems(op, sh):
    if op == wl.OP_CONV:
        P, Q = synthdata.conv_out_hw(sh[2], sh[3], sh[5], sh[6], sh[7], sh[8])
        return sh[0] * sh[4] * P * Q
    return sh[0] * sh[1]


def first_reach(L):
    """{instance: (task name, op, shape, key)} over the tasks, smallest
    problem first, and the set of instances per family."""
    tasks = sorted(all_tasks(), key=lambda t: (wl.flops(t[1], t[2]), t[0]))
    first = {}
    for name, op, sh in tasks:
        keys, inst, _ = L.Space(op, sh).programs()
        uniq, pos = np.unique(inst, return_index=True)
        for i, p in zip(uniq.tolist(), pos.tolist()):
            if i not in first:
                first[i] = (name, op, sh, int(keys[p]))
    return first


def test_every_reachable_instance_bit_exact_and_within_its_budget(env):
    torch, L = env
    first = first_reach(L)
    by_task = collections.defaultdict(list)
    for inst, (name, op, sh, key) in first.items():
        by_task[(name, op, sh)].append((inst, key))
    tested = collections.Counter()
    reach = collections.Counter(FAMILY[i // 4096] for i in first)
    for (name, op, sh), items in sorted(by_task.items(), key=lambda t: wl.flops(t[0][1], t[0][2])):
        if op == wl.OP_CONV:
            x, w = synthdata.conv_inputs(sh, "int")
        else:
            x, w = synthdata.matmul_inputs(sh, "int")
        n = out_elems(op, sh)
        xd = torch.from_numpy(np.ascontiguousarray(x)).cuda()
        wd = torch.from_numpy(np.ascontiguousarray(w)).cuda()
        yb = torch.empty(n + TAIL, dtype=torch.float32, device="cuda:0")
        rng = np.random.default_rng(len(items))
        idx = np.unique(np.concatenate([rng.integers(0, n, 400), [0, n - 1]])).astype(np.int64)
        ref = (ok.conv2d_f64_points(x, w, sh, idx) if op == wl.OP_CONV
               else ok.matmul_f64_points(x, w, idx))
        idx_d = torch.from_numpy(idx).cuda()
        space = L.Space(op, sh)
        print(f"{name}: {len(items)} instances", flush=True)
        for inst, key in sorted(items):
            pt = space.from_key(key)
            info = space.kernel_info(pt, with_attrs=True)
            what = f"{name} {FAMILY[info['family']]}{info['params']} {space.knobs(pt)}"
            assert info["instance"] == inst
            assert info["local_bytes"] == 0, f"{what}: spills {info['local_bytes']} B per lane"
            assert info["max_threads_per_block"] >= info["threads"], what
            assert info["static_lds_bytes"] + info["lds_bytes"] <= LDS_LIMIT, what
            yb[:n].fill_(float("nan"))
            yb[n:].fill_(CANARY)
            L.kernel_run(op, space.sched(pt), xd, wd, yb)
            torch.cuda.synchronize()
            assert bool(torch.isfinite(yb[:n]).all()), f"{what}: unwritten or non-finite output"
            assert bool((yb[n:] == CANARY).all()), f"{what}: write past the end"
            got = yb[:n][idx_d].cpu().numpy().astype(np.float64)
            assert np.array_equal(got, ref), f"{what}: differs from the oracle"
            tested[FAMILY[info["family"]]] += 1
        del xd, wd, yb
    for fam in sorted(reach):
        print(f"{fam}: reachable {reach[fam]}, tested {tested[fam]}", flush=True)
    assert tested == reach
    assert sum(reach.values()) == len(first) > 1000


@pytest.mark.parametrize("name,op,sh", all_tasks(), ids=[t[0] for t in all_tasks()])
def test_tuned_winner_full_output(env, name, op, sh):
    """A short tuning run (the combined approach with 30 samples and a
    Droplet budget of 10) at the workload's size; its winner matches the oracle
    on every output within the tolerance."""
    torch, L = env
    kind = "uniform" if name in wl.SINGLE else "he"
    if op == wl.OP_CONV:
        x, w = synthdata.conv_inputs(sh, kind)
        ref = ok.conv2d_f64(x, w, sh).ravel()
    else:
        x, w = synthdata.matmul_inputs(sh, kind)
        ref = ok.matmul_f64(x, w).ravel()
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y = torch.empty(ref.size, dtype=torch.float32, device="cuda:0")
    space = L.Space(op, sh)
    cfg = L.tune_cfg(n_explore=30, budget=10, seed=wl.BASE_SEED + 7,
                     measure=L.measure_cfg(repeat=5, min_repeat_ms=0.2))
    res, _ = L.ds_tune(space, cfg, L.make_io(xd, wd, y))
    print(name, space.knobs(res.best), f"{res.best_ms * 1e3:.1f} us", flush=True)
    y.fill_(float("nan"))
    L.kernel_run(op, res.best, xd, wd, y)
    torch.cuda.synchronize()
    got = y.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(got))
    scale = float(np.abs(ref).max())
    assert float(np.abs(got - ref).max()) <= 1e-4 * scale
