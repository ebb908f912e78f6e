"""Pins of the fp64 conv2d / matmul oracle against facts that do not come from it.

* closed form for all-ones tensors (count of in-bounds taps times C);
* delta weights reproduce a shifted input channel exactly;
* a pure-Python loop nest on tiny shapes, an independent numpy im2col GEMM and
  torch's float64 conv2d (a library routine) agree with it;
* matmul: all-ones gives K, identity gives A, numpy's float64 matmul agrees.
"""
import itertools

import numpy as np
import pytest
import torch

import synthdata
from oracle import kernels as ok


def taps(p, n_in, R, st, pd):
    """In-bounds taps of output row p: |{r < R : 0 <= p*st - pd + r < n_in}|."""
    lo = max(0, pd - p * st)
    hi = min(R, n_in + pd - p * st)
    return max(0, hi - lo)


@pytest.mark.parametrize(
    "shape",
    [
        (1, 64, 56, 56, 64, 3, 3, 1, 1),
        (1, 3, 224, 224, 4, 7, 7, 2, 3),
        (2, 5, 9, 7, 3, 3, 2, 2, 1),
        (1, 4, 28, 28, 2, 1, 1, 2, 0),
    ],
)
def test_conv_all_ones_closed_form(shape):
    N, C, H, W, K, R, S, st, pd = shape
    x, w = synthdata.conv_inputs(shape, "ones")
    y = ok.conv2d_f64(x, w, shape)
    P, Q = y.shape[2:]
    ch = np.array([taps(p, H, R, st, pd) for p in range(P)], np.float64)
    cw = np.array([taps(q, W, S, st, pd) for q in range(Q)], np.float64)
    expect = C * ch[:, None] * cw[None, :]
    assert np.array_equal(y, np.broadcast_to(expect, y.shape))


def test_conv_all_ones_named_values():
    # 56x56, 3x3, stride 1, pad 1, C=64: corners see 4 taps, edges 6, interior 9.
    y = ok.conv2d_f64(*synthdata.conv_inputs((1, 64, 56, 56, 2, 3, 3, 1, 1), "ones"),
                      (1, 64, 56, 56, 2, 3, 3, 1, 1))
    assert sorted(set(y.ravel().tolist())) == [256.0, 384.0, 576.0]
    assert y[0, 0, 0, 0] == 256 and y[0, 1, 0, 5] == 384 and y[0, 0, 5, 5] == 576
    # 224x224, 7x7, stride 2, pad 3, C=3 -> 112x112; row taps 4,6,7,...,7,5.
    sh = (1, 3, 224, 224, 1, 7, 7, 2, 3)
    y = ok.conv2d_f64(*synthdata.conv_inputs(sh, "ones"), sh)
    assert y.shape == (1, 1, 112, 112)
    assert y[0, 0, 0, 0] == 48 and y[0, 0, 50, 50] == 147 and y[0, 0, 111, 111] == 75
    assert y[0, 0, 1, 0] == 3 * 6 * 4


@pytest.mark.parametrize("r0,s0", [(0, 0), (0, 2), (2, 1), (1, 1)])
def test_conv_delta_weights_shift(r0, s0):
    sh = (2, 3, 8, 9, 3, 3, 3, 1, 1)
    N, C, H, W, K, R, S, st, pd = sh
    x = synthdata.uniform(7, (N, C, H, W))
    w = np.zeros((K, C, R, S), np.float32)
    for k in range(K):
        w[k, k % C, r0, s0] = 1.0
    y = ok.conv2d_f64(x, w, sh)
    xp = np.zeros((N, C, H + 2, W + 2), np.float32)
    xp[:, :, 1:-1, 1:-1] = x
    for k in range(K):
        expect = xp[:, k % C, r0:r0 + H, s0:s0 + W]
        assert np.array_equal(y[:, k], expect.astype(np.float64))


def brute_conv(x, w, sh):
    N, C, H, W, K, R, S, st, pd = sh
    P = (H + 2 * pd - R) // st + 1
    Q = (W + 2 * pd - S) // st + 1
    y = [[[[0.0] * Q for _ in range(P)] for _ in range(K)] for _ in range(N)]
    for n in range(N):
        for k in range(K):
            for p in range(P):
                for q in range(Q):
                    acc = 0.0
                    for c in range(C):
                        for r in range(R):
                            for s in range(S):
                                iy, ix = p * st - pd + r, q * st - pd + s
                                if 0 <= iy < H and 0 <= ix < W:
                                    acc += float(x[n, c, iy, ix]) * float(w[k, c, r, s])
                    y[n][k][p][q] = acc
    return np.array(y, np.float64)


def im2col_conv(x, w, sh):
    N, C, H, W, K, R, S, st, pd = sh
    P = (H + 2 * pd - R) // st + 1
    Q = (W + 2 * pd - S) // st + 1
    xp = np.zeros((N, C, H + 2 * pd, W + 2 * pd), np.float64)
    xp[:, :, pd:pd + H, pd:pd + W] = x
    cols = np.empty((N, C, R, S, P, Q), np.float64)
    for r in range(R):
        for s in range(S):
            cols[:, :, r, s] = xp[:, :, r:r + st * (P - 1) + 1:st, s:s + st * (Q - 1) + 1:st]
    cols = cols.reshape(N, C * R * S, P * Q)
    wm = w.astype(np.float64).reshape(K, C * R * S)
    return np.einsum("kc,ncp->nkp", wm, cols).reshape(N, K, P, Q)


def tiny_shapes():
    rng = np.random.default_rng(2406)
    out = []
    for _ in range(40):
        R, S = int(rng.integers(1, 4)), int(rng.integers(1, 5))
        st, pd = int(rng.integers(1, 4)), int(rng.integers(0, 3))
        H, W = int(rng.integers(R, 8)), int(rng.integers(S, 8))
        out.append((int(rng.integers(1, 3)), int(rng.integers(1, 4)), H, W,
                    int(rng.integers(1, 4)), R, S, st, pd))
    return out


@pytest.mark.parametrize("sh", tiny_shapes())
def test_conv_brute_force_and_library(sh):
    x = synthdata.uniform(11, sh[:4])
    w = synthdata.uniform(12, (sh[4], sh[1], sh[5], sh[6]))
    y = ok.conv2d_f64(x, w, sh)
    scale = max(1.0, np.abs(y).max())
    assert np.abs(y - brute_conv(x, w, sh)).max() <= 1e-12 * scale
    assert np.abs(y - im2col_conv(x, w, sh)).max() <= 1e-12 * scale
    yt = torch.nn.functional.conv2d(torch.from_numpy(x).double(), torch.from_numpy(w).double(),
                                    stride=sh[7], padding=sh[8]).numpy()
    assert np.abs(y - yt).max() <= 1e-12 * scale


def test_conv_points_match_full():
    sh = (2, 5, 13, 11, 6, 3, 3, 2, 1)
    x, w = synthdata.conv_inputs(sh, "uniform", seed=5)
    y = ok.conv2d_f64(x, w, sh)
    idx = np.array([0, 1, 17, y.size // 2, y.size - 1], np.int64)
    assert np.array_equal(ok.conv2d_f64_points(x, w, sh, idx), y.ravel()[idx])
    with pytest.raises(ValueError):
        ok.conv2d_f64_points(x, w, sh, np.array([y.size], np.int64))


def test_conv_integer_inputs_exact():
    # Small integers: every partial sum is an integer below 2**53, so the
    # oracle is exact and must equal integer arithmetic.
    sh = (1, 16, 10, 10, 4, 3, 3, 1, 1)
    x, w = synthdata.conv_inputs(sh, "int")
    y = ok.conv2d_f64(x, w, sh)
    xi = x.astype(np.int64)
    wi = w.astype(np.int64)
    ref = np.zeros(y.shape, np.int64)
    xp = np.zeros((1, 16, 12, 12), np.int64)
    xp[:, :, 1:-1, 1:-1] = xi
    for k in range(4):
        for c in range(16):
            for r in range(3):
                for s in range(3):
                    ref[0, k] += wi[k, c, r, s] * xp[0, c, r:r + 10, s:s + 10]
    assert np.array_equal(y, ref.astype(np.float64))


def test_conv_rejects_empty_output():
    with pytest.raises(ValueError):
        ok.conv_out((1, 1, 2, 2, 1, 5, 5, 1, 0))


def test_matmul_pins():
    M, N, K = 37, 53, 1024
    A, B = synthdata.matmul_inputs((M, N, K), "ones")
    assert np.array_equal(ok.matmul_f64(A, B), np.full((M, N), float(K)))
    A = synthdata.uniform(3, (M, 41))
    I = np.eye(41, dtype=np.float32)
    assert np.array_equal(ok.matmul_f64(A, I), A.astype(np.float64))
    A, B = synthdata.matmul_inputs((M, N, 300), "uniform")
    C = ok.matmul_f64(A, B)
    ref = A.astype(np.float64) @ B.astype(np.float64)
    assert np.abs(C - ref).max() <= 1e-12 * np.abs(ref).max()
    # Element by element on a non-square product (catches transposed operands).
    A = synthdata.uniform(4, (3, 5))
    B = synthdata.uniform(5, (5, 2))
    C = ok.matmul_f64(A, B)
    for i, j in itertools.product(range(3), range(2)):
        assert C[i, j] == pytest.approx(sum(float(A[i, l]) * float(B[l, j]) for l in range(5)),
                                        abs=1e-14)
    idx = np.array([0, 5, 5], np.int64)
    assert np.array_equal(ok.matmul_f64_points(A, B, idx), C.ravel()[idx])


def test_matmul_empty_rows():
    A = np.zeros((0, 8), np.float32)
    B = synthdata.uniform(1, (8, 4))
    assert ok.matmul_f64(A, B).shape == (0, 4)
