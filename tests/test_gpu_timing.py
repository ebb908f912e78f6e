"""Timing sanity of the measurement harness (Section 2.1: a measured schedule
stands for its running time).

For fixed schedules of the five workload families (the small convolution and
matmul, the strided 7x7 stem, a batch-1 ResNet-50 layer at 32 reduction
splits, a VGG-16 layer over band tiles), each timed as the tuner times it:
  * the implied rate never exceeds the chip: algorithmic flop / median time
    <= 157.3 TFLOP/s (fp32 dense peak of MI355X);
  * the repeats are consistent: min <= median <= every repeat's max, the
    spread (max / min of the repeats) stays under 1.5, and a second
    measurement of the same point lands within 15% of the first;
  * every launch is slower than the empty-kernel floor.
"""
import pytest

import synthdata
from synthdata import workloads as wl

pytestmark = pytest.mark.gpu

PEAK_FLOPS = 157.3e12


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a device"
    return torch


@pytest.fixture(scope="module")
def lib(torch_dev):
    from paper_2406_20037_amd import _lib
    return _lib


CASES = [
    ("conv3x3_c64_56", None,
     dict(tk=16, th=4, tw=16, tc=64, unroll=64, lds=1, ks=2, mfma=2, vec=4)),
    ("matmul_1024", None,
     dict(bm=64, bn=64, bk=16, unroll=64, dbuf=1, mfma=1, ks=1, vec=4)),
    ("conv7x7_s2_c3_224", None,
     dict(tk=16, th=8, tw=16, tc=1, unroll=16, lds=1, ks=1, mfma=1, vec=4)),
    ("resnet50", "s4_3x3_512_512_s2",
     dict(tk=32, th=8, tw=4, tc=16, unroll=0, lds=1, ks=32, mfma=3, vec=4)),
    ("vgg16", "L6_256_256_56",
     dict(tk=64, th=4, tw=64, tc=8, unroll=64, lds=1, ks=4, mfma=3, vec=4)),
]


def setup_case(torch, L, workload, layer):
    if layer is None:
        op, sh = wl.SINGLE[workload]
        kind = "uniform"
    else:
        table = {"resnet50": wl.RESNET50, "vgg16": wl.VGG16}[workload]
        op, sh = next((o, s) for name, o, s, _ in table if name == layer)
        kind = "he"
    if op == wl.OP_CONV:
        x, w = synthdata.conv_inputs(sh, kind)
        P, Q = synthdata.conv_out_hw(sh[2], sh[3], sh[5], sh[6], sh[7], sh[8])
        n = sh[0] * sh[4] * P * Q
    else:
        x, w = synthdata.matmul_inputs(sh, kind)
        n = sh[0] * sh[1]
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y, ref = torch.empty(n, device="cuda:0"), torch.empty(n, device="cuda:0")
    L.kernel_run_reference(op, sh, xd, wd, ref)
    torch.cuda.synchronize()
    return op, sh, L.make_io(xd, wd, y, ref), (xd, wd, y, ref)


@pytest.mark.parametrize("workload,layer,knobs", CASES, ids=[c[1] or c[0] for c in CASES])
def test_timing_is_physical_and_stable(torch_dev, lib, workload, layer, knobs):
    torch, L = torch_dev, lib
    op, sh, io, keep = setup_case(torch, L, workload, layer)
    space = L.Space(op, sh)
    s = space.sched_of(**knobs)
    assert space.valid(s.index())
    print("timing", workload, layer, knobs, flush=True)
    cfg = L.measure_cfg(repeat=11)
    a = L.ds_measure(s, io, cfg)
    b = L.ds_measure(s, io, cfg)
    floor = L.ds_empty_kernel_floor()
    for m in (a, b):
        assert m.status == 0 and m.nonfinite == 0
        assert m.max_err <= 1e-4 * m.max_ref
        reps = [m.repeats_ms[i] for i in range(m.n_repeats)]
        assert m.n_repeats == 11 and min(reps) == m.min_ms
        assert m.min_ms <= m.median_ms <= max(reps)
        assert max(reps) / m.min_ms < 1.5, reps
        assert m.median_ms > floor.median_ms
        rate = wl.flops(op, sh) / (m.median_ms * 1e-3)
        assert rate <= PEAK_FLOPS, f"{rate / 1e12:.1f} TFLOP/s exceeds the fp32 peak"
    assert abs(a.median_ms - b.median_ms) <= 0.15 * min(a.median_ms, b.median_ms)
    del keep


def test_mfma_ceiling_is_physical(torch_dev, lib):
    """The pure-MFMA calibration launch: a rate under the published fp32 peak
    and above half of it, its median at its fastest repeats."""
    torch, L = torch_dev, lib
    sink = torch.empty(L.DS_MFMA_CEILING_SINK, device="cuda:0")
    print("mfma ceiling", flush=True)
    m, flop = L.ds_mfma_ceiling(sink, iters=512, cfg=L.measure_cfg(repeat=7))
    torch.cuda.synchronize()
    assert m.status == 0 and m.n_repeats == 7
    assert flop == 1024 * 4 * 512 * 16 * 2048
    rate = flop / (m.median_ms * 1e-3)
    assert 0.5 * PEAK_FLOPS < rate <= PEAK_FLOPS, f"{rate / 1e12:.1f} TFLOP/s"
    # single host launches: an occasional slow one, but the median sits at
    # the fast ones
    assert m.median_ms <= 1.1 * m.min_ms, [m.repeats_ms[i] for i in range(m.n_repeats)]
    assert bool(torch.isfinite(sink).all())
