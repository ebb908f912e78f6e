"""fp64 conv2d / matmul oracle: ctypes wrapper over ``oracle_kernels.c``.

Test infrastructure only (see the package header).  The C file states the
definitions (ONNX / TVM ``conv2d_nchw`` reading of the paper's conv2d kernel,
Section 3 RQ6, and row-major matmul).

Pins (tests/test_oracle_kernels.py): closed form for all-ones inputs, delta
weights (pure shift), a pure-Python loop nest on tiny shapes, an independent
numpy im2col GEMM, and ``torch.nn.functional.conv2d`` in float64.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle_kernels.c")
LIB = os.path.join(HERE, "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (-O3 -fopenmp, no fast-math)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O3", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", SRC, "-o", tmp]
        )
        os.replace(tmp, LIB)
    return LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        lib = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        i64 = ctypes.c_int64
        lib.oracle_conv2d_f64.argtypes = [P, P, P, P]
        lib.oracle_conv2d_f64_points.argtypes = [P, P, P, P, i64, P]
        lib.oracle_conv2d_out.argtypes = [P, P, P]
        lib.oracle_matmul_f64.argtypes = [P, P, P, i64, i64, i64]
        lib.oracle_matmul_f64_points.argtypes = [P, P, i64, i64, i64, P, i64, P]
        lib.oracle_num_threads.argtypes = []
        for f in (lib.oracle_conv2d_f64, lib.oracle_conv2d_f64_points, lib.oracle_conv2d_out,
                  lib.oracle_matmul_f64, lib.oracle_matmul_f64_points, lib.oracle_num_threads):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _f32(a) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a


def conv_out(shape9):
    sh = np.asarray(shape9, dtype=np.int64)
    P = np.zeros(1, np.int64)
    Q = np.zeros(1, np.int64)
    if _load().oracle_conv2d_out(_ptr(sh), _ptr(P), _ptr(Q)) != 0:
        raise ValueError(f"conv shape has no output: {tuple(shape9)}")
    return int(P[0]), int(Q[0])


def conv2d_f64(x, w, shape9) -> np.ndarray:
    """y[N,K,P,Q] (float64) for x[N,C,H,W], w[K,C,R,S] under shape9."""
    N, C, H, W, K, R, S, st, pd = (int(v) for v in shape9)
    x = _f32(x)
    w = _f32(w)
    assert x.shape == (N, C, H, W) and w.shape == (K, C, R, S)
    P, Q = conv_out(shape9)
    y = np.empty((N, K, P, Q), np.float64)
    sh = np.asarray(shape9, dtype=np.int64)
    rc = _load().oracle_conv2d_f64(_ptr(x), _ptr(w), _ptr(y), _ptr(sh))
    if rc != 0:
        raise ValueError("oracle_conv2d_f64 rejected the shape")
    return y


def conv2d_f64_points(x, w, shape9, idx) -> np.ndarray:
    x = _f32(x)
    w = _f32(w)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.size, np.float64)
    sh = np.asarray(shape9, dtype=np.int64)
    rc = _load().oracle_conv2d_f64_points(_ptr(x), _ptr(w), _ptr(sh), _ptr(idx), idx.size, _ptr(out))
    if rc != 0:
        raise ValueError("oracle_conv2d_f64_points: bad shape or index")
    return out


def matmul_f64(A, B) -> np.ndarray:
    A = _f32(A)
    B = _f32(B)
    M, K = A.shape
    K2, N = B.shape
    assert K == K2
    C = np.empty((M, N), np.float64)
    rc = _load().oracle_matmul_f64(_ptr(A), _ptr(B), _ptr(C), M, N, K)
    if rc != 0:
        raise ValueError("oracle_matmul_f64 rejected the shape")
    return C


def matmul_f64_points(A, B, idx) -> np.ndarray:
    A = _f32(A)
    B = _f32(B)
    M, K = A.shape
    N = B.shape[1]
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.size, np.float64)
    rc = _load().oracle_matmul_f64_points(_ptr(A), _ptr(B), M, N, K, _ptr(idx), idx.size, _ptr(out))
    if rc != 0:
        raise ValueError("oracle_matmul_f64_points: bad shape or index")
    return out


def num_threads() -> int:
    return int(_load().oracle_num_threads())
