"""Split-reduction workspaces are per (device, stream).

Two split schedules queued on two streams with no ordering between them must
both be right (they no longer share partials); a split schedule can be
captured into a HIP graph on a stream whose workspace already exists, and a
capture on a stream without one is refused before anything is recorded.
"""
import numpy as np
import pytest

import synthdata
from oracle import kernels as ok

pytestmark = pytest.mark.gpu

TOL = 1e-4


@pytest.fixture(scope="module")
def env():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a device"
    from paper_2406_20037_amd import _lib
    return torch, _lib


def conv_case(torch, L, sh, knobs):
    x, w = synthdata.conv_inputs(sh, "uniform")
    ref = ok.conv2d_f64(x, w, sh).ravel()
    space = L.Space(L.DS_OP_CONV2D_NCHW, sh)
    s = space.sched_of(**knobs)
    assert space.valid(s.index()) and knobs["ks"] > 1
    return dict(s=s, ref=ref, x=torch.from_numpy(x).cuda(), w=torch.from_numpy(w).cuda(),
                y=torch.full((ref.size,), float("nan"), device="cuda:0"))


def close(torch, c):
    y = c["y"].cpu().numpy().astype(np.float64)
    scale = float(np.abs(c["ref"]).max())
    assert np.all(np.isfinite(y))
    assert float(np.abs(y - c["ref"]).max()) <= TOL * scale


def test_two_streams_split_concurrently(env):
    torch, L = env
    a = conv_case(torch, L, (1, 64, 40, 40, 64, 3, 3, 1, 1),
                  dict(tk=16, th=4, tw=32, tc=16, unroll=0, lds=1, ks=4, mfma=1, vec=4))
    b = conv_case(torch, L, (2, 32, 24, 24, 48, 3, 3, 1, 1),
                  dict(tk=16, th=4, tw=8, tc=8, unroll=0, lds=1, ks=2, mfma=1, vec=4))
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    print("two streams", flush=True)
    for _ in range(3):
        L.kernel_run(L.DS_OP_CONV2D_NCHW, a["s"], a["x"], a["w"], a["y"], s1)
        L.kernel_run(L.DS_OP_CONV2D_NCHW, b["s"], b["x"], b["w"], b["y"], s2)
    torch.cuda.synchronize()
    close(torch, a)
    close(torch, b)


SPLIT_CASES = [
    ((1, 64, 40, 40, 64, 3, 3, 1, 1),
     dict(tk=16, th=4, tw=32, tc=16, unroll=0, lds=1, ks=4, mfma=1, vec=4)),
    # channel-quad family, band tiles, four splits across workgroups
    ((2, 32, 14, 14, 64, 3, 3, 1, 1),
     dict(tk=32, th=4, tw=16, tc=4, unroll=0, lds=1, ks=4, mfma=3, vec=4)),
    # rectangular tiles, two wave groups and two splits across workgroups
    ((1, 64, 40, 40, 64, 3, 3, 1, 1),
     dict(tk=16, th=4, tw=16, tc=8, unroll=0, lds=1, ks=4, mfma=2, vec=4)),
]


@pytest.mark.parametrize("sh,knobs", SPLIT_CASES, ids=["mfma1", "mfma2_band", "mfma2_kg2"])
def test_capture_after_the_workspace_exists(env, sh, knobs):
    """Graph replays of a captured split schedule (main kernel and reduce
    launch) give the eager result bit for bit, on both MFMA conv families."""
    torch, L = env
    c = conv_case(torch, L, sh, knobs)
    st = torch.cuda.Stream()
    # first call outside capture creates this stream's workspace
    L.kernel_run(L.DS_OP_CONV2D_NCHW, c["s"], c["x"], c["w"], c["y"], st)
    torch.cuda.synchronize()
    close(torch, c)
    eager = c["y"].clone()
    g = torch.cuda.CUDAGraph()
    print("capture", flush=True)
    with torch.cuda.graph(g, stream=st):
        L.kernel_run(L.DS_OP_CONV2D_NCHW, c["s"], c["x"], c["w"], c["y"], st)
    for _ in range(3):
        c["y"].fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(c["y"], eager), "graph replay differs from the eager launch"
    del g


MANY_SPLITS = [
    # band tiles, 32 splits of 64 quad chunks (stride 2)
    ((1, 256, 14, 14, 64, 3, 3, 2, 1),
     dict(tk=16, th=2, tw=8, tc=4, unroll=0, lds=1, ks=32, mfma=3, vec=4)),
    # rectangular tiles, 1x1 filter, 32 splits
    ((1, 512, 7, 7, 64, 1, 1, 1, 0),
     dict(tk=16, th=4, tw=4, tc=4, unroll=0, lds=1, ks=32, mfma=2, vec=4)),
    # tabled MFMA family, 32 splits
    ((1, 256, 14, 14, 64, 3, 3, 2, 1),
     dict(tk=16, th=4, tw=4, tc=4, unroll=0, lds=1, ks=32, mfma=1, vec=4)),
    # VALU family: 24 chunks over 16 splits leave 4 of them empty (12 partials)
    ((1, 96, 7, 7, 32, 3, 3, 1, 1),
     dict(tk=4, th=4, tw=4, tc=4, unroll=0, lds=1, ks=16, mfma=0, vec=4)),
]


@pytest.mark.parametrize("sh,knobs", MANY_SPLITS,
                         ids=["band_ks32", "rect_ks32", "mfma1_ks32", "valu_ks16_empty"])
def test_many_splits_match_the_oracle(env, sh, knobs):
    """16 and 32 reduction splits (a reduce launch over as many partial
    slices, empty splits skipped) agree with the fp64 oracle."""
    torch, L = env
    c = conv_case(torch, L, sh, knobs)
    splits = L.Space(L.DS_OP_CONV2D_NCHW, sh).kernel_info(c["s"].index())["splits"]
    assert splits == (12 if sh[1] == 96 else knobs["ks"])
    print("many splits", sh, knobs, flush=True)
    L.kernel_run(L.DS_OP_CONV2D_NCHW, c["s"], c["x"], c["w"], c["y"], torch.cuda.current_stream())
    torch.cuda.synchronize()
    close(torch, c)


def test_capture_without_a_workspace_is_refused(env):
    torch, L = env
    c = conv_case(torch, L, (1, 32, 20, 20, 32, 3, 3, 1, 1),
                  dict(tk=16, th=4, tw=16, tc=4, unroll=0, lds=1, ks=8, mfma=1, vec=4))
    st = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    err = None
    print("refused capture", flush=True)
    try:
        with torch.cuda.graph(g, stream=st):
            try:
                L.kernel_run(L.DS_OP_CONV2D_NCHW, c["s"], c["x"], c["w"], c["y"], st)
            except RuntimeError as e:      # raised before anything is recorded
                err = e
            c["y"].zero_()                 # keeps the captured graph non-empty
    finally:
        torch.cuda.synchronize()
    assert err is not None and "DS_EUNSUPPORTED" in str(err)
