"""Host-side checks of the C-ABI library against the oracle (no GPU needed).

Integer bookkeeping (value lists, validity, geometry, keys, neighbours, the
sampler's draw sequence, Droplet's trace with a supplied cost) must agree with
the oracle bit for bit.
"""
import math
import re

import numpy as np
import pytest

import synthdata
from synthdata import workloads as wl
from oracle import droplet as odr
from oracle import sampler as osm
from oracle import space as osp

lib = pytest.importorskip("paper_2406_20037_amd._lib")

ALL_SHAPES = ([(op, sh) for op, sh in wl.SINGLE.values()]
              + [(op, sh) for _, op, sh, _ in wl.RESNET50]
              + [(op, sh) for _, op, sh, _ in wl.VGG16])

ODD_SHAPES = [
    (1, (2, 3, 9, 7, 5, 3, 2, 2, 1)),
    (1, (1, 1, 1, 1, 1, 1, 1, 1, 0)),
    (1, (3, 17, 13, 11, 33, 5, 5, 3, 2)),
    (1, (0, 4, 8, 8, 4, 3, 3, 1, 1)),
    (2, (3, 5, 2)),
    (2, (0, 64, 64)),
    (2, (129, 67, 300)),
    (2, (1, 1, 1)),
]


def header_functions():
    text = open(lib.HERE + "/../include/droplet.h").read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^(?:const\s+char\s*\*|int|void)\s*\*?\s*([a-z_][a-z0-9_]*)\s*\(",
                       text, flags=re.M)
    return sorted(set(names))


def test_library_exports_every_declared_function():
    names = header_functions()
    assert len(names) >= 25
    for n in names:
        assert hasattr(lib.lib, n), n
    assert set(names) == set(lib.SIGNATURES), set(names) ^ set(lib.SIGNATURES)
    assert lib.ds_num_instances() > 1000


def test_fail_loudly_without_library(tmp_path, monkeypatch):
    import importlib.util
    spec = importlib.util.spec_from_file_location("lib_copy", lib.__file__)
    mod = importlib.util.module_from_spec(spec)
    monkeypatch.setattr("os.path.exists", lambda p: False)
    with pytest.raises(RuntimeError, match="no CPU fallback"):
        spec.loader.exec_module(mod)


def both(op, sh):
    return lib.Space(op, sh), osp.Space(op, sh)


@pytest.mark.parametrize("op,sh", ALL_SHAPES + ODD_SHAPES)
def test_space_matches_oracle(op, sh):
    c, o = both(op, sh)
    assert c.values == o.values and c.names == o.names and c.size == o.size()
    assert c.origin() == o.origin()
    rng = np.random.default_rng(abs(hash((op, sh))) % 2 ** 32)
    n = o.size()
    keys = range(n) if n <= 3000 else rng.choice(n, 1500, replace=False)
    for k in keys:
        k = int(k)
        idx = o.from_key(k)
        assert c.from_key(k) == idx and c.key(idx) == k
        assert c.valid(idx) == o.valid(idx)
        assert c.geometry(idx) == o.geometry(idx), (idx, o.knobs(idx))
        assert c.neighbors(idx) == o.neighbors(idx)


@pytest.mark.parametrize("op,sh", list(wl.SINGLE.values()) + ODD_SHAPES)
def test_every_valid_point_has_a_kernel(op, sh):
    c, o = both(op, sh)
    pts = o.valid_points()
    if len(pts) > 20000:
        pts = pts[:: len(pts) // 20000 + 1]
    missing = [p for p in pts if not c.has_kernel(p)]
    assert not missing, [o.knobs(p) for p in missing[:5]]


@pytest.mark.parametrize("op,sh", [(op, sh) for _, op, sh, _ in wl.RESNET50 + wl.VGG16])
def test_model_layers_have_kernels(op, sh):
    c, o = both(op, sh)
    rng = np.random.default_rng(7)
    for k in rng.choice(o.size(), 600, replace=False):
        p = o.from_key(int(k))
        if o.valid(p):
            assert c.has_kernel(p), o.knobs(p)


@pytest.mark.parametrize("op,sh", list(wl.SINGLE.values()) + [(1, (2, 3, 9, 7, 5, 3, 2, 2, 1))])
@pytest.mark.parametrize("seed", [0, 1, 17, 240620037])
def test_sampler_sequence_bit_exact(op, sh, seed):
    c, o = both(op, sh)
    assert c.draw(seed, 300) == osm.sample(o, seed, 300)


def test_sampler_small_lattice_and_exhaustion():
    vals = [[0, 1, 2, 3], [0, 1, 2], [5, 6]]
    inv = [1, 5, 7, 20]
    c = lib.Space(lattice=vals, invalid_keys=inv)
    o = osp.Lattice(vals, predicate=lambda p: osp.Lattice(vals).key(p) not in inv)
    for seed in range(30):
        assert c.draw(seed, 10) == osm.sample(o, seed, 10)
    assert sorted(c.draw(3, 300)) == sorted(o.valid_points())
    allbad = lib.Space(lattice=[[0, 1]], invalid_keys=[0, 1])
    assert allbad.draw(1, 5) == []


def test_example3_trace_through_c_abi(golden_dir):
    vals = [[1, 2, 3, 4, 5], [1, 2, 4, 8, 16]]
    c = lib.Space(lattice=vals)
    assert c.neighbors((2, 3)) == [(1, 3), (3, 3), (2, 2), (2, 4)]

    def cost(idx):
        u, t = vals[0][idx[0]], vals[1][idx[1]]
        return (u - 4) ** 2 + (math.log2(t) - 1) ** 2

    cfg = lib.tune_cfg(alpha=1.0)
    res, trace = lib.droplet_tune_ex(c, None, 100, cfg, None, cost, trace_cap=64)
    path_rows = [l.split()[1:] for l in open(f"{golden_dir}/droplet_trace_example3.txt")
                 if l.startswith("order")][0]
    order = [tuple(int(v) for v in s.split(",")) for s in path_rows]
    got = [tuple(vals[a][i] for a, i in enumerate(c.from_key(t[2]))) for t in trace]
    assert got == order
    assert res.best.index() == (3, 1) and res.n_droplet_measured == 11 and res.best_ms == 0
    assert res.n_moves == 4 and res.status == 0


def random_cost_table(space, seed, noisy=False):
    rng = np.random.default_rng(seed)
    table = {}

    def cost(idx):
        if idx not in table:
            base = float(rng.uniform(1.0, 2.0))
            table[idx] = [base * float(rng.uniform(0.97, 1.03)) for _ in range(11)] if noisy else base
        return table[idx]

    return cost


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("alpha", [1.0, 0.05])
def test_droplet_matches_oracle_on_conv_space(seed, alpha):
    op, sh = wl.SINGLE["conv3x3_c64_56"]
    c, o = both(op, sh)
    smooth = lambda p: [float(sum((i - 2) ** 2 * (a + 1) for a, i in enumerate(p))) + 1.0 + 0.01 * r
                        for r in range(11)] if alpha < 1 else float(sum((i - 2) ** 2 * (a + 1) for a, i in enumerate(p)))
    start = o.valid_points()[seed * 997]
    ref = odr.droplet(o, smooth, start=start, budget=100, alpha=alpha)
    res, trace = lib.droplet_tune_ex(c, start, 100, lib.tune_cfg(alpha=alpha), None, smooth,
                                     trace_cap=256)
    assert res.best.index() == ref["best"]
    assert [t[2] for t in trace] == ref["order"]
    assert res.n_droplet_measured == ref["measured"]
    assert (res.status == 0) == (ref["status"] == odr.OK)


@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("noisy", [False, True])
def test_combined_matches_oracle(seed, noisy):
    op, sh = wl.SINGLE["matmul_1024"]
    c, o = both(op, sh)
    alpha = 0.05 if noisy else 1.0
    cost_o = random_cost_table(o, seed, noisy)
    ref = odr.combined(o, cost_o, seed=seed, n_explore=300, budget=100, alpha=alpha)
    cost_c = random_cost_table(o, seed, noisy)
    res, trace = lib.ds_tune(c, lib.tune_cfg(alpha=alpha, seed=seed), None, cost_c, trace_cap=512)
    assert res.n_explore_measured == ref["n_explore"] == 300
    assert res.seed_point.index() == ref["seed_point"]
    assert res.best.index() == ref["best"]
    assert res.n_droplet_measured == ref["n_droplet"]
    assert [t[2] for t in trace[:300]] == [o.key(p) for p in ref["samples"]]


def test_budget_and_failures_through_c_abi():
    vals = [list(range(6)), list(range(6))]
    c = lib.Space(lattice=vals)
    cost = lambda p: None if p == (1, 0) else float((p[0] - 5) ** 2 + (p[1] - 5) ** 2)
    res, trace = lib.droplet_tune_ex(c, (0, 0), 3, lib.tune_cfg(alpha=1.0), None, cost, trace_cap=16)
    assert res.status == lib.DS_EBUDGET and res.n_droplet_measured == 4
    assert res.n_failed == 1 and trace[1][1] != 0 and math.isinf(trace[1][3])
    o = osp.Lattice(vals)
    ocost = lambda p: math.inf if p == (1, 0) else float((p[0] - 5) ** 2 + (p[1] - 5) ** 2)
    ref = odr.droplet(o, ocost, start=(0, 0), budget=3)
    assert res.best.index() == ref["best"] and [t[2] for t in trace] == ref["order"]


def test_budget_stop_mid_neighbourhood_through_c_abi():
    """The budget runs out inside a neighbourhood after a faster neighbour was
    measured: the search still moves there (the hand-worked case of the
    oracle's budget pin on Example 3's lattice)."""
    vals = [[1, 2, 3, 4, 5], [1, 2, 4, 8, 16]]
    c = lib.Space(lattice=vals)
    o = osp.Lattice(vals)
    cost = lambda p: float((vals[0][p[0]] - 4) ** 2 + (math.log2(vals[1][p[1]]) - 1) ** 2)
    for budget, best in ((2, (1, 0)), (3, (2, 0))):
        res, trace = lib.droplet_tune_ex(c, (0, 0), budget, lib.tune_cfg(alpha=1.0), None, cost,
                                         trace_cap=16)
        ref = odr.droplet(o, cost, start=(0, 0), budget=budget)
        assert res.status == lib.DS_EBUDGET and ref["status"] == odr.EBUDGET
        assert res.best.index() == ref["best"] == best
        assert [t[2] for t in trace] == ref["order"]
        assert res.best_ms == ref["meas"].median


def test_frozen_axes_through_c_abi():
    vals = [list(range(4)), [0, 1]]
    c = lib.Space(lattice=vals)
    cost = lambda p: float((p[0] - 3) ** 2 + (0 if p[1] == 1 else 5))
    res, _ = lib.droplet_tune_ex(c, (0, 0), 100, lib.tune_cfg(alpha=1.0, frozen_mask=2), None, cost)
    assert res.best.index() == (3, 0)
    res, _ = lib.droplet_tune_ex(c, (0, 0), 100, lib.tune_cfg(alpha=1.0), None, cost)
    assert res.best.index() == (3, 1)


def test_gen_uniform_matches_synthdata():
    for seed in (0, 240620037, 240620038):
        buf = lib.ds_gen_uniform(seed, 5000)
        assert np.array_equal(np.ctypeslib.as_array(buf), synthdata.uniform(seed, (5000,)))


def test_error_paths_without_gpu():
    with pytest.raises(lib.DsError, match="DS_EINVAL"):
        lib.Space(1, (1, 0, 4, 4, 1, 3, 3, 1, 1))
    with pytest.raises(lib.DsError, match="DS_EINVAL"):
        lib.Space(1, (1, 1, 2, 2, 1, 5, 5, 1, 0))
    with pytest.raises(lib.DsError, match="DS_EUNSUPPORTED"):
        lib.Space(3, (4, 4, 4))
    with pytest.raises(lib.DsError, match="DS_EUNSUPPORTED"):
        lib.Space(2, (1 << 20, 1 << 20, 4))
    s = lib.Space(1, wl.SINGLE["conv3x3_c64_56"][1])
    o = osp.Space(1, wl.SINGLE["conv3x3_c64_56"][1])
    bad = next(p for p in (o.from_key(k) for k in range(o.size())) if not o.valid(p))
    with pytest.raises(lib.DsError, match="DS_EINVALID_SCHED"):
        lib.kernel_run(1, s.sched(bad), 0, 0, 0, 0)
    with pytest.raises(lib.DsError, match="DS_EINVAL"):
        s.from_key(s.size)
    assert not s.valid((99,) + (0,) * 7)                    # outside the lattice
    with pytest.raises(lib.DsError, match="DS_EINVAL"):
        s.key((99,) + (0,) * 7)
    m = lib.Space(2, (8, 8, 8))
    with pytest.raises(lib.DsError, match="DS_EINVAL"):
        lib.kernel_run(2, s.sched(s.origin()), 0, 0, 0, 0)    # op mismatch
    with pytest.raises(lib.DsError, match="DS_EINVAL"):
        lib.droplet_tune_ex(m, None, 10, None, None, None)   # GPU mode needs buffers


class _FakeSink:
    """Stands for a device tensor: an address and an element count (the
    argument checks run before anything touches the device)."""
    def __init__(self, n, addr=0x10000):
        self.n, self.addr = n, addr

    def data_ptr(self):
        return self.addr

    def numel(self):
        return self.n


def test_mfma_ceiling_argument_errors_without_gpu():
    with pytest.raises(lib.DsError, match="DS_EINVAL"):
        lib.ds_mfma_ceiling(_FakeSink(lib.DS_MFMA_CEILING_SINK, addr=0))     # null sink
    with pytest.raises(lib.DsError, match="DS_EINVAL"):
        lib.ds_mfma_ceiling(_FakeSink(lib.DS_MFMA_CEILING_SINK - 1))        # sink too small
    with pytest.raises(lib.DsError, match="DS_EINVAL"):
        lib.ds_mfma_ceiling(_FakeSink(lib.DS_MFMA_CEILING_SINK), iters=0)


def test_single_hip_runtime_in_process():
    """Loading the binding first must not map a second HIP runtime next to torch's."""
    import subprocess
    import sys
    code = ("import paper_2406_20037_amd as p; p._lib.ds_num_instances(); import torch, re; "
            "print(len(set(re.findall(r'/\\S*libamdhip64\\S*', open('/proc/self/maps').read()))))")
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                         cwd=lib.HERE + "/..", timeout=300)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip().splitlines()[-1] == "1"


def test_degenerate_tuning_cases():
    """The method's degenerate cases through the C ABI and in the oracle:
    nothing to explore, nothing valid, an exploration that exhausts the
    lattice, a Droplet start at the origin when the origin is invalid, and a
    zero Droplet budget."""
    vals = [list(range(3)), list(range(4))]
    pred = lambda p: (p[0] + p[1]) % 3 != 0          # (0, 0) is invalid
    o = osp.Lattice(vals, predicate=pred)
    inv = [k for k in range(o.size()) if not o.valid(o.from_key(k))]
    c = lib.Space(lattice=vals, invalid_keys=inv)
    cost = lambda p: float((p[0] - 2) ** 2 + (p[1] - 1) ** 2 + 0.1 * p[1])

    # no exploration budget: nothing to hand to Droplet Search
    assert odr.combined(o, cost, seed=1, n_explore=0)["status"] == odr.EEXHAUSTED
    with pytest.raises(lib.DsError) as e:
        lib.ds_tune(c, lib.tune_cfg(n_explore=0, seed=1), None, cost)
    assert e.value.rc == lib.DS_EEXHAUSTED

    # a lattice without a valid point
    dead = osp.Lattice(vals, predicate=lambda p: False)
    cd = lib.Space(lattice=vals, invalid_keys=list(range(dead.size())))
    assert odr.combined(dead, cost, seed=1, n_explore=5)["status"] == odr.EEXHAUSTED
    with pytest.raises(lib.DsError) as e:
        lib.ds_tune(cd, lib.tune_cfg(n_explore=5, seed=1), None, cost)
    assert e.value.rc == lib.DS_EEXHAUSTED

    # exploring more points than the lattice holds measures every valid point
    # once; Droplet then finds every neighbour cached and stops at the optimum
    nvalid = len(o.valid_points())
    ref = odr.combined(o, cost, seed=2, n_explore=50)
    res, _ = lib.ds_tune(c, lib.tune_cfg(n_explore=50, seed=2, alpha=1.0), None, cost)
    assert res.n_explore_measured == ref["n_explore"] == nvalid
    assert res.best.index() == ref["best"] == min(o.valid_points(), key=cost)
    assert res.n_droplet_measured == ref["n_droplet"] == 0

    # Droplet from "no optimisation": the origin is invalid, so the first
    # valid point in key order
    ref = odr.droplet(o, cost, start=None, budget=100)
    res, trace = lib.droplet_tune_ex(c, None, 100, lib.tune_cfg(alpha=1.0), None, cost,
                                     trace_cap=64)
    assert ref["path"][0] == o.origin() == (1, 0)
    assert res.seed_point.index() == (1, 0)
    assert res.best.index() == ref["best"] and [t[2] for t in trace] == ref["order"]

    # a zero budget measures the start only
    ref = odr.droplet(o, cost, start=(1, 0), budget=0)
    res, _ = lib.droplet_tune_ex(c, (1, 0), 0, lib.tune_cfg(alpha=1.0), None, cost)
    assert ref["status"] == odr.EBUDGET and res.status == lib.DS_EBUDGET
    assert res.n_droplet_measured == ref["measured"] == 1 and res.best.index() == (1, 0)
