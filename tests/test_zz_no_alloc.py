"""kernel_run_noalloc through the C ABI against kernel_run on the same inputs.

The entry point launches the same kernels as kernel_run but keeps split
partials in a fixed device array, so on every split schedule its output must
equal kernel_run's bit for bit, and both must meet the oracle's tolerance
(max |y - ref| <= 1e-4 * max |ref|).  Two calls in a row, the second on a
smaller problem, check that the array's leftover contents never leak into a
result; a schedule whose partials exceed the array is refused before launch.
"""
import numpy as np
import pytest

import synthdata
from oracle import kernels as ok
from oracle import space as osp

pytestmark = pytest.mark.gpu

TOL = 1e-4


@pytest.fixture(scope="module")
def env():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a device"
    from paper_2406_20037_amd import _lib
    return torch, _lib


def run_both(torch, L, op, sh, knobs, kind="uniform"):
    if op == L.DS_OP_CONV2D_NCHW:
        x, w = synthdata.conv_inputs(sh, kind)
        ref = ok.conv2d_f64(x, w, sh).ravel()
    else:
        x, w = synthdata.matmul_inputs(sh, kind)
        ref = ok.matmul_f64(x, w).ravel()
    space = L.Space(op, sh)
    s = space.sched_of(**knobs)
    assert space.valid(s.index()), knobs
    xd = torch.from_numpy(x).cuda()
    wd = torch.from_numpy(w).cuda()
    ya = torch.full((ref.size,), float("nan"), device="cuda:0")
    yb = torch.full((ref.size,), float("nan"), device="cuda:0")
    L.kernel_run(op, s, xd, wd, ya)
    torch.cuda.synchronize()
    print(f"noalloc {op} {sh} {knobs}", flush=True)
    L.kernel_run_noalloc(op, s, xd, wd, yb)
    torch.cuda.synchronize()
    a = ya.cpu().numpy()
    b = yb.cpu().numpy()
    assert np.all(np.isfinite(b))
    assert np.array_equal(a, b), "kernel_run_noalloc differs from kernel_run"
    scale = float(np.abs(ref).max())
    err = float(np.abs(b.astype(np.float64) - ref).max())
    assert err <= TOL * scale, f"max err {err:.3g} vs max ref {scale:.3g}"


CONV_BIG = ((1, 64, 56, 56, 64, 3, 3, 1, 1),
            dict(tk=16, th=4, tw=32, tc=32, unroll=16, lds=1, ks=2, mfma=1, vec=4))
CONV_SMALL = ((1, 48, 13, 11, 40, 3, 3, 1, 1),
              dict(tk=16, th=4, tw=8, tc=4, unroll=0, lds=1, ks=4, mfma=1, vec=4))
MM_BIG = ((256, 512, 1024), dict(bm=64, bn=64, bk=32, unroll=16, dbuf=1, mfma=1, ks=4, vec=4))
MM_SMALL = ((33, 45, 70), dict(bm=16, bn=16, bk=8, unroll=0, dbuf=0, mfma=0, ks=8, vec=1))


def test_two_calls_conv_then_smaller(env):
    torch, L = env
    run_both(torch, L, L.DS_OP_CONV2D_NCHW, *CONV_BIG)
    run_both(torch, L, L.DS_OP_CONV2D_NCHW, *CONV_SMALL)


def test_two_calls_matmul_then_smaller(env):
    torch, L = env
    run_both(torch, L, L.DS_OP_MATMUL_RM, *MM_BIG)
    run_both(torch, L, L.DS_OP_MATMUL_RM, *MM_SMALL)


def test_unsplit_schedule_needs_no_scratch(env):
    torch, L = env
    run_both(torch, L, L.DS_OP_CONV2D_NCHW, (1, 3, 30, 30, 64, 7, 7, 2, 3),
             dict(tk=16, th=4, tw=8, tc=1, unroll=0, lds=1, ks=1, mfma=1, vec=1))


def test_partials_beyond_the_array_are_refused(env):
    torch, L = env
    # VGG-16 layer 2 at batch 16: 16*64*224*224 outputs, two splits -> 102.8M floats
    sh = (16, 64, 224, 224, 64, 3, 3, 1, 1)
    space = L.Space(L.DS_OP_CONV2D_NCHW, sh)
    s = space.sched_of(tk=64, th=4, tw=16, tc=16, unroll=0, lds=1, ks=2, mfma=1, vec=4)
    assert space.valid(s.index())
    P, Q = osp.conv_out(sh)
    assert 2 * sh[0] * sh[4] * P * Q > L.DS_NOALLOC_MAX_FLOATS
    x = torch.zeros(sh[0] * sh[1] * sh[2] * sh[3], device="cuda:0")
    w = torch.zeros(sh[4] * sh[1] * 9, device="cuda:0")
    y = torch.full((sh[0] * sh[4] * P * Q,), 7.0, device="cuda:0")
    with pytest.raises(RuntimeError, match="DS_EINVAL"):
        L.kernel_run_noalloc(L.DS_OP_CONV2D_NCHW, s, x, w, y)
    torch.cuda.synchronize()
    assert float(y[:1024].min()) == 7.0 and float(y[-1024:].max()) == 7.0, "refused call wrote y"
