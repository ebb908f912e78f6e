"""Seeded synthetic inputs shared by the CPU oracle and the HIP path.

This module holds no arithmetic of the tuning method or of the kernels: it only
turns a seed into reproducible fp32 tensors.  The generator is SplitMix64
(Steele, Lea and Flood, "Fast splittable pseudorandom number generators",
OOPSLA 2014): the i-th output (i = 0, 1, ...) of stream ``seed`` is
``mix(seed + (i + 1) * 0x9E3779B97F4A7C15 mod 2**64)`` with the published
two-multiply finaliser.  Because the generator is counter based, any element
can be regenerated on its own.

Distributions:

* ``uniform``: ``u = (z >> 40) * 2**-24``, ``v = 2u - 1``; every value is exact
  in fp32 and lies in [-1, 1).
* ``normal``: Box-Muller on two consecutive outputs in fp64
  (``u1 = ((z1 >> 11) + 1) * 2**-53`` in (0, 1], ``u2 = (z2 >> 11) * 2**-53``),
  scaled by ``sigma`` and rounded once to fp32.
* ``small_int``: integers in [-a, a] drawn as ``((z >> 32) * (2a+1)) >> 32``
  minus ``a``; stored as fp32 (exact).
* ``he_normal``: ``normal`` with ``sigma = sqrt(2 / fan_in)``.

Seeds: ``BASE_SEED`` plus a per-tensor offset (x: +0, w: +1, B or third
tensor: +2).
"""
from __future__ import annotations

import math

import numpy as np

BASE_SEED = 240620037
GAMMA = np.uint64(0x9E3779B97F4A7C15)
M1 = np.uint64(0xBF58476D1CE4E5B9)
M2 = np.uint64(0x94D049BB133111EB)


def splitmix64(seed: int, n: int, start: int = 0) -> np.ndarray:
    """Outputs ``start .. start+n-1`` of the SplitMix64 stream ``seed`` (uint64)."""
    idx = np.arange(start + 1, start + n + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(seed % (1 << 64)) + idx * GAMMA
        z = (z ^ (z >> np.uint64(30))) * M1
        z = (z ^ (z >> np.uint64(27))) * M2
        z = z ^ (z >> np.uint64(31))
    return z


def uniform(seed: int, shape) -> np.ndarray:
    n = int(np.prod(shape))
    z = splitmix64(seed, n)
    u = (z >> np.uint64(40)).astype(np.float64) * (2.0 ** -24)
    return (2.0 * u - 1.0).astype(np.float32).reshape(shape)


def normal(seed: int, shape, sigma: float = 1.0) -> np.ndarray:
    n = int(np.prod(shape))
    z = splitmix64(seed, 2 * n)
    u1 = ((z[0::2] >> np.uint64(11)).astype(np.float64) + 1.0) * (2.0 ** -53)
    u2 = (z[1::2] >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)
    v = np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * math.pi * u2)
    return (sigma * v).astype(np.float32).reshape(shape)


def he_normal(seed: int, shape, fan_in: int) -> np.ndarray:
    return normal(seed, shape, math.sqrt(2.0 / fan_in))


def small_int(seed: int, shape, a: int) -> np.ndarray:
    n = int(np.prod(shape))
    z = splitmix64(seed, n) >> np.uint64(32)
    with np.errstate(over="ignore"):
        v = (z * np.uint64(2 * a + 1)) >> np.uint64(32)
    return (v.astype(np.int64) - a).astype(np.float32).reshape(shape)


def conv_out_hw(H, W, R, S, stride, pad):
    return (H + 2 * pad - R) // stride + 1, (W + 2 * pad - S) // stride + 1


def conv_inputs(shape, kind: str = "uniform", seed: int = BASE_SEED):
    """x[N,C,H,W], w[K,C,R,S] for a conv shape (N,C,H,W,K,R,S,stride,pad)."""
    N, C, H, W, K, R, S, st, pd = shape
    if kind == "uniform":
        return uniform(seed, (N, C, H, W)), uniform(seed + 1, (K, C, R, S))
    if kind == "he":
        return normal(seed, (N, C, H, W)), he_normal(seed + 1, (K, C, R, S), C * R * S)
    if kind == "int":
        return small_int(seed, (N, C, H, W), 8), small_int(seed + 1, (K, C, R, S), 2)
    if kind == "ones":
        return np.ones((N, C, H, W), np.float32), np.ones((K, C, R, S), np.float32)
    raise ValueError(kind)


def matmul_inputs(shape, kind: str = "uniform", seed: int = BASE_SEED):
    """A[M,K], B[K,N] for a matmul shape (M,N,K)."""
    M, N, K = shape
    if kind == "uniform":
        return uniform(seed, (M, K)), uniform(seed + 2, (K, N))
    if kind == "he":
        return normal(seed, (M, K)), he_normal(seed + 2, (K, N), K)
    if kind == "int":
        return small_int(seed, (M, K), 8), small_int(seed + 2, (K, N), 2)
    if kind == "ones":
        return np.ones((M, K), np.float32), np.ones((K, N), np.float32)
    raise ValueError(kind)
