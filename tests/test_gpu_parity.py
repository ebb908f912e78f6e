"""GPU parity of the HIP kernel family against the fp64 oracle, through the C ABI.

Bar: max |y - ref| <= 1e-4 * max |ref| for U[-1,1) and He-normal inputs; exact
equality for small-integer and all-ones inputs (every partial sum is an
integer below 2**24, so every fp32 summation order is exact).  Outputs are
NaN-prefilled (catches unwritten outputs) and followed by a canary tail
(catches writes past the end).
"""
import zlib

import numpy as np
import pytest

import synthdata
from synthdata import workloads as wl
from oracle import kernels as ok
from oracle import space as osp

pytestmark = pytest.mark.gpu

TOL = 1e-4
CANARY = 12345.0
TAIL = 64


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a device"
    return torch


@pytest.fixture(scope="module")
def lib(torch_dev):
    from paper_2406_20037_amd import _lib
    return _lib


def to_dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")


def out_elems(op, sh):
    if op == 1:
        P, Q = osp.conv_out(sh)
        return sh[0] * sh[4] * P * Q
    return sh[0] * sh[1]


class Runner:
    def __init__(self, torch, lib, op, sh, x, w):
        self.torch, self.lib, self.op, self.sh = torch, lib, op, sh
        self.space = lib.Space(op, sh)
        self.x, self.w = to_dev(torch, x), to_dev(torch, w)
        self.n = out_elems(op, sh)
        self.ybuf = torch.empty(self.n + TAIL, dtype=torch.float32, device="cuda:0")

    def run(self, idx):
        t = self.torch
        self.ybuf[: self.n].fill_(float("nan"))
        self.ybuf[self.n:].fill_(CANARY)
        self.lib.kernel_run(self.op, self.space.sched(idx), self.x, self.w, self.ybuf)
        t.cuda.synchronize()
        out = self.ybuf.cpu().numpy()
        assert np.all(out[self.n:] == CANARY), "write past the end of y"
        return out[: self.n].astype(np.float64)


def pick_points(o, n_random, seed, per_value=2):
    """Random valid points plus, for every axis value, a few valid points
    taking it (so every knob value is exercised)."""
    rng = np.random.default_rng(seed)
    pts = set()
    size = o.size()
    tries = 0
    while len(pts) < n_random and tries < 100 * n_random:
        tries += 1
        p = o.from_key(int(rng.integers(size)))
        if o.valid(p):
            pts.add(p)
    for a, n in enumerate(o.sizes):
        for v in range(n):
            got, tries = 0, 0
            while got < per_value and tries < 4000:
                tries += 1
                p = list(o.from_key(int(rng.integers(size))))
                p[a] = v
                p = tuple(p)
                if o.valid(p):
                    pts.add(p)
                    got += 1
    return sorted(pts)


def check_close(y, ref, what):
    scale = np.abs(ref).max()
    err = np.abs(y - ref).max() if y.size else 0.0
    assert np.all(np.isfinite(y)), f"{what}: non-finite output"
    assert err <= TOL * scale, f"{what}: max err {err:.3g} vs max ref {scale:.3g}"


PARITY_CASES = [
    ("conv3x3_c64_56", 1, (1, 64, 56, 56, 64, 3, 3, 1, 1), 220),
    ("conv7x7_s2_c3_224", 1, (1, 3, 224, 224, 64, 7, 7, 2, 3), 160),
    ("matmul_1024", 2, (1024, 1024, 1024), 160),
    ("conv_ragged", 1, (2, 5, 19, 23, 7, 3, 3, 2, 1), 250),
    ("conv_ragged_5x5", 1, (1, 37, 15, 13, 40, 5, 5, 1, 2), 200),
    ("conv_1x1_s2", 1, (1, 24, 17, 17, 48, 1, 1, 2, 0), 150),
    ("matmul_ragged", 2, (129, 67, 300), 250),
    ("matmul_fc", 2, (1, 1000, 2048), 120),
    ("matmul_k_odd", 2, (33, 45, 7), 150),
    ("conv_7x7_out", 1, (2, 32, 7, 7, 48, 3, 3, 1, 1), 200),
]


@pytest.mark.parametrize("name,op,sh,n", PARITY_CASES, ids=[c[0] for c in PARITY_CASES])
def test_parity_uniform(torch_dev, lib, name, op, sh, n):
    if op == 1:
        x, w = synthdata.conv_inputs(sh, "uniform")
        ref = ok.conv2d_f64(x, w, sh).ravel()
    else:
        x, w = synthdata.matmul_inputs(sh, "uniform")
        ref = ok.matmul_f64(x, w).ravel()
    r = Runner(torch_dev, lib, op, sh, x, w)
    o = osp.Space(op, sh)
    pts = pick_points(o, n, seed=zlib.crc32(name.encode()) % 1000)
    for p in pts:
        print(name, o.knobs(p), flush=True)
        check_close(r.run(p), ref, f"{name} {o.knobs(p)}")


EXACT_CASES = [
    ("conv3x3_c64_56", 1, (1, 64, 56, 56, 64, 3, 3, 1, 1)),
    ("conv_ragged", 1, (2, 5, 19, 23, 7, 3, 3, 2, 1)),
    ("conv7x7_s2", 1, (1, 3, 60, 60, 16, 7, 7, 2, 3)),
    ("matmul_ragged", 2, (129, 67, 300)),
    ("matmul_256", 2, (256, 256, 512)),
    ("conv_7x7_out", 1, (2, 32, 7, 7, 48, 3, 3, 1, 1)),
]


@pytest.mark.parametrize("kind", ["int", "ones"])
@pytest.mark.parametrize("name,op,sh", EXACT_CASES, ids=[c[0] for c in EXACT_CASES])
def test_parity_bit_exact(torch_dev, lib, name, op, sh, kind):
    if op == 1:
        x, w = synthdata.conv_inputs(sh, kind)
        ref = ok.conv2d_f64(x, w, sh).ravel()
    else:
        x, w = synthdata.matmul_inputs(sh, kind)
        ref = ok.matmul_f64(x, w).ravel()
    assert np.abs(ref).max() < 2 ** 24
    r = Runner(torch_dev, lib, op, sh, x, w)
    o = osp.Space(op, sh)
    for p in pick_points(o, 80, seed=3, per_value=1):
        y = r.run(p)
        assert np.array_equal(y, ref), f"{name} {kind} {o.knobs(p)}"


def test_matmul_every_mfma_class_exact(torch_dev, lib):
    """One point of every MFMA matmul class (tile, K-tile, stages, split and
    the two operand-prefetch depths) on an aligned shape, where full tiles take
    the direct, software-pipelined path: bit-exact on small-integer inputs."""
    sh = (256, 256, 512)
    x, w = synthdata.matmul_inputs(sh, "int")
    ref = ok.matmul_f64(x, w).ravel()
    r = Runner(torch_dev, lib, 2, sh, x, w)
    o = osp.Space(2, sh)
    seen = set()
    for p in o.valid_points():
        k = o.knobs(p)
        if k["mfma"] != 1:
            continue
        cls = (k["bm"], k["bn"], k["bk"], k["dbuf"], k["ks"], k["unroll"] >= 16, k["vec"])
        if cls in seen:
            continue
        seen.add(cls)
        y = r.run(p)
        assert np.array_equal(y, ref), f"matmul {sh} int {k}"
    assert len(seen) > 500


@pytest.mark.parametrize("shift_x,shift_w", [(1, 0), (0, 1), (1, 1)])
def test_parity_misaligned_operands(torch_dev, lib, shift_x, shift_w):
    """Operands that start 4 bytes past a 16-byte boundary: the 16-byte staging
    copies (weights, aligned halo rows, direct matmul tiles) must give way to
    the 4-byte ones without changing the result.  Small-integer inputs, so
    every schedule must match the oracle exactly."""
    torch = torch_dev

    def shifted(a, k):
        buf = torch.zeros(a.size + k, dtype=torch.float32, device="cuda:0")
        buf[k:] = torch.from_numpy(np.ascontiguousarray(a).ravel()).to("cuda:0")
        return buf[k:]

    cases = [(1, (1, 64, 56, 56, 64, 3, 3, 1, 1)), (1, (1, 3, 224, 224, 64, 7, 7, 2, 3)),
             (2, (256, 256, 512))]
    for op, sh in cases:
        if op == 1:
            x, w = synthdata.conv_inputs(sh, "int")
            ref = ok.conv2d_f64(x, w, sh).ravel()
        else:
            x, w = synthdata.matmul_inputs(sh, "int")
            ref = ok.matmul_f64(x, w).ravel()
        xd, wd = shifted(x, shift_x), shifted(w, shift_w)
        assert (xd.data_ptr() % 16 == 0) == (shift_x == 0)
        n = out_elems(op, sh)
        y = torch.empty(n, dtype=torch.float32, device="cuda:0")
        space = lib.Space(op, sh)
        o = osp.Space(op, sh)
        pts = [p for p in pick_points(o, 60, seed=11, per_value=1)
               if o.knobs(p).get("lds", 1) == 1 or op == 2]
        for p in pts:
            y.fill_(float("nan"))
            lib.kernel_run(op, space.sched(p), xd, wd, y)
            torch.cuda.synchronize()
            out = y.cpu().numpy().astype(np.float64)
            assert np.array_equal(out, ref), f"{sh} shift x {shift_x} w {shift_w} {o.knobs(p)}"


@pytest.mark.parametrize("mfma,th,tw", [(2, 16, 16), (3, 8, 16)], ids=["rect_4x4", "band_4x2"])
def test_register_budget_follows_copy_width(torch_dev, lib, mfma, th, tw):
    """A point whose 16-byte copies need at most 4 units per thread runs the
    channel-quad build that holds 4 copy sources in registers; on operands 4
    bytes past a 16-byte boundary the same point copies 4 bytes at a time,
    needs more units and runs the 12-unit build.  Eight chunks per workgroup,
    so the held sources are reused; both runs match the oracle exactly."""
    torch = torch_dev
    sh = (2, 32, 28, 28, 64, 3, 3, 1, 1)
    kn = dict(tk=64, th=th, tw=tw, tc=4, unroll=0, lds=1, ks=1, mfma=mfma, vec=4)
    space = lib.Space(1, sh)
    s16, s4 = space.sched_of(**kn), space.sched_of(**dict(kn, vec=1))
    assert space.valid(s16.index()) and space.valid(s4.index())
    assert space.kernel_info(s16.index())["params"][4] == 4
    assert space.kernel_info(s4.index())["params"][4] == 12
    x, w = synthdata.conv_inputs(sh, "int")
    ref = ok.conv2d_f64(x, w, sh).ravel()
    y = torch.empty(ref.size, dtype=torch.float32, device="cuda:0")
    def shifted(a, k):
        buf = torch.zeros(a.size + k, dtype=torch.float32, device="cuda:0")
        buf[k:] = torch.from_numpy(np.ascontiguousarray(a).ravel()).to("cuda:0")
        return buf[k:]

    for shift in (0, 1):
        xd, wd = shifted(x, shift), shifted(w, shift)
        assert (xd.data_ptr() % 16 == 0) == (wd.data_ptr() % 16 == 0) == (shift == 0)
        print("register budget", mfma, th, tw, "shift", shift, flush=True)
        y.fill_(float("nan"))
        lib.kernel_run(1, s16, xd, wd, y)
        torch.cuda.synchronize()
        assert np.array_equal(y.cpu().numpy().astype(np.float64), ref), f"shift {shift}"


BAND_CASES = [
    ("band_14_cross", (2, 16, 14, 14, 32, 3, 3, 1, 1)),
    ("band_7_multi", (3, 8, 7, 7, 16, 3, 3, 1, 1)),
    ("band_1x1_s2", (1, 16, 56, 56, 32, 1, 1, 2, 0)),
    ("band_3x3_s2", (2, 16, 28, 28, 16, 3, 3, 2, 1)),
    ("band_c3_7x7_s2", (2, 3, 20, 20, 16, 7, 7, 2, 3)),
    ("band_odd", (2, 12, 13, 13, 20, 3, 3, 1, 1)),
    ("band_pad0", (2, 20, 9, 9, 24, 3, 3, 1, 0)),
    ("band_5x5", (2, 4, 30, 30, 17, 5, 5, 1, 2)),
    ("band_wide", (1, 8, 5, 40, 16, 3, 3, 1, 1)),
]


@pytest.mark.parametrize("name,sh", BAND_CASES, ids=[c[0] for c in BAND_CASES])
def test_parity_band_tiles(torch_dev, lib, name, sh):
    """mfma = 3 band tiles (runs of consecutive output pixels across rows and
    images): small-integer inputs, so every schedule must match the oracle
    exactly; every output written and nothing past the end.  Half the points
    also run on operands 4 bytes past a 16-byte boundary."""
    torch = torch_dev
    x, w = synthdata.conv_inputs(sh, "int")
    ref = ok.conv2d_f64(x, w, sh).ravel()
    r = Runner(torch_dev, lib, 1, sh, x, w)
    o = osp.Space(1, sh)
    pts = [p for p in o.valid_points() if o.knobs(p)["mfma"] == 3]
    assert pts
    rng = np.random.default_rng(zlib.crc32(name.encode()) % 1000)
    if len(pts) > 120:
        pts = [pts[i] for i in sorted(rng.choice(len(pts), 120, replace=False))]
    xs = torch.zeros(x.size + 1, dtype=torch.float32, device="cuda:0")
    xs[1:] = torch.from_numpy(np.ascontiguousarray(x).ravel()).to("cuda:0")
    ws = torch.zeros(w.size + 1, dtype=torch.float32, device="cuda:0")
    ws[1:] = torch.from_numpy(np.ascontiguousarray(w).ravel()).to("cuda:0")
    y = torch.empty(ref.size, dtype=torch.float32, device="cuda:0")
    space = lib.Space(1, sh)
    for i, p in enumerate(pts):
        print(name, o.knobs(p), flush=True)
        assert np.array_equal(r.run(p), ref), f"{name} {o.knobs(p)}"
        if i % 2:
            y.fill_(float("nan"))
            lib.kernel_run(1, space.sched(p), xs[1:], ws[1:], y)
            torch.cuda.synchronize()
            out = y.cpu().numpy().astype(np.float64)
            assert np.array_equal(out, ref), f"{name} misaligned {o.knobs(p)}"


def test_empty_batch_and_rows(torch_dev, lib):
    torch = torch_dev
    s = lib.Space(1, (0, 4, 8, 8, 4, 3, 3, 1, 1))
    lib.kernel_run(1, s.sched(s.origin()), 0, 0, 0)
    m = lib.Space(2, (0, 64, 64))
    x = torch.zeros(1, device="cuda:0")
    lib.kernel_run(2, m.sched(m.origin()), x, x, x)
    torch.cuda.synchronize()


def test_reference_kernels(torch_dev, lib):
    torch = torch_dev
    for op, sh in [(1, (2, 5, 19, 23, 7, 3, 3, 2, 1)), (2, (129, 67, 300))]:
        if op == 1:
            x, w = synthdata.conv_inputs(sh, "uniform")
            ref = ok.conv2d_f64(x, w, sh).ravel()
        else:
            x, w = synthdata.matmul_inputs(sh, "uniform")
            ref = ok.matmul_f64(x, w).ravel()
        y = torch.empty(ref.size, device="cuda:0")
        lib.kernel_run_reference(op, sh, to_dev(torch, x), to_dev(torch, w), y)
        torch.cuda.synchronize()
        check_close(y.cpu().numpy().astype(np.float64), ref, f"reference {sh}")


MODEL_SCHEDULES = [
    dict(tk=32, th=8, tw=8, tc=16, unroll=64, lds=1, ks=1, mfma=1, vec=4),
    dict(tk=16, th=4, tw=16, tc=8, unroll=16, lds=1, ks=2, mfma=1, vec=4),
    dict(tk=8, th=4, tw=8, tc=8, unroll=16, lds=1, ks=1, mfma=0, vec=1),
    dict(tk=16, th=8, tw=8, tc=4, unroll=0, lds=0, ks=1, mfma=1, vec=1),
    dict(tk=64, th=8, tw=32, tc=16, unroll=512, lds=1, ks=1, mfma=2, vec=4),
    dict(tk=64, th=4, tw=64, tc=8, unroll=16, lds=1, ks=2, mfma=3, vec=4),
]


def nearest_valid(o, want):
    """The valid point closest (breadth-first in index steps) to the point
    whose knob values are nearest to want."""
    target = tuple(v.index(want[n]) if want[n] in v else
                   min(range(len(v)), key=lambda i: abs(np.log2(max(1, v[i])) -
                                                        np.log2(max(1, want[n]))))
                   for v, n in zip(o.values, o.names))
    seen, frontier = {target}, [target]
    while frontier:
        for p in frontier:
            if o.valid(p):
                return p
        nxt = []
        for p in frontier:
            for a in range(len(p)):
                for d in (-1, 1):
                    q = p[:a] + (p[a] + d,) + p[a + 1:]
                    if 0 <= q[a] < o.sizes[a] and q not in seen:
                        seen.add(q)
                        nxt.append(q)
        frontier = nxt
    return None


@pytest.mark.parametrize("name,op,sh,count", wl.RESNET50 + wl.VGG16,
                         ids=[l[0] for l in wl.RESNET50] + ["vgg_" + l[0] for l in wl.VGG16])
def test_model_layers_sampled(torch_dev, lib, name, op, sh, count):
    """Full-size layers: sampled outputs against the oracle's one-by-one sums."""
    if op == 1:
        x, w = synthdata.conv_inputs(sh, "he")
    else:
        x, w = synthdata.matmul_inputs(sh, "he")
    r = Runner(torch_dev, lib, op, sh, x, w)
    o = osp.Space(op, sh)
    rng = np.random.default_rng(11)
    idx = np.unique(np.concatenate([rng.integers(0, r.n, 3000), [0, r.n - 1]])).astype(np.int64)
    ref = ok.conv2d_f64_points(x, w, sh, idx) if op == 1 else ok.matmul_f64_points(x, w, idx)
    scheds = MODEL_SCHEDULES if op == 1 else [
        dict(bm=16, bn=64, bk=64, unroll=64, dbuf=1, mfma=0, ks=8, vec=4),
        dict(bm=16, bn=16, bk=16, unroll=16, dbuf=0, mfma=0, ks=1, vec=1)]
    seen = set()
    for want in scheds:
        p = nearest_valid(o, want)
        if p in seen:
            continue
        seen.add(p)
        print(name, o.knobs(p), flush=True)
        y = r.run(p)
        assert np.all(np.isfinite(y)), f"{name} {o.knobs(p)}: unwritten or non-finite output"
        check_close(y[idx], ref, f"{name} {o.knobs(p)}")


def test_measure_and_parity_detection(torch_dev, lib):
    torch = torch_dev
    op, sh = wl.SINGLE["conv3x3_c64_56"]
    x, w = synthdata.conv_inputs(sh, "uniform")
    ref = ok.conv2d_f64(x, w, sh).astype(np.float32).ravel()
    s = lib.Space(op, sh)
    xd, wd = to_dev(torch, x), to_dev(torch, w)
    y = torch.empty(ref.size, device="cuda:0")
    good = to_dev(torch, ref)
    io = lib.make_io(xd, wd, y, good)
    p = s.sched_of(tk=32, th=8, tw=8, tc=16, unroll=64, lds=1, ks=1, mfma=1, vec=4)
    m = lib.ds_measure(p, io, lib.measure_cfg(repeat=7))
    assert m.status == 0 and m.n_repeats == 7 and 0 < m.median_ms < 10
    assert m.max_err <= 1e-4 * m.max_ref and m.nonfinite == 0
    bad = to_dev(torch, ref + 1.0)
    io_bad = lib.make_io(xd, wd, y, bad)
    m = lib.ds_measure(p, io_bad, lib.measure_cfg(repeat=3))
    assert m.status == lib.DS_EPARITY
    floor = lib.ds_empty_kernel_floor()
    assert 0 < floor.median_ms < 0.1


def test_tune_small_budget(torch_dev, lib):
    torch = torch_dev
    op, sh = wl.SINGLE["conv3x3_c64_56"]
    x, w = synthdata.conv_inputs(sh, "uniform")
    s = lib.Space(op, sh)
    y = torch.empty(out_elems(op, sh), device="cuda:0")
    io = lib.make_io(to_dev(torch, x), to_dev(torch, w), y)
    cfg = lib.tune_cfg(n_explore=24, budget=12, measure=lib.measure_cfg(repeat=5, min_repeat_ms=0.1))
    res, trace = lib.ds_tune(s, cfg, io, trace_cap=128)
    assert res.n_explore_measured == 24 and res.n_droplet_measured <= 12
    assert res.best_ms <= res.seed_ms and res.n_failed == 0
    assert all(t[1] == 0 for t in trace)
    o = osp.Space(op, sh)
    assert o.valid(res.best.index())
    best, ms = lib.droplet_tune(2, (64, 64, 64), None, 6)
    assert ms > 0 and osp.Space(2, (64, 64, 64)).valid(best.index())
