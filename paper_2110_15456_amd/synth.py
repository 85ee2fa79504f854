"""Seeded synthetic inputs (numpy PCG64), shared by the tests, the oracle
checks and the benchmark.  This module holds no BFP arithmetic: it only draws
FP32 arrays with the shapes and value distributions of the workloads.

Distributions (draws in float64, rounded once to float32):
  half_normal     |N(0, 1)|           ReLU activations
  weights         N(0, 0.02)          weights
  grads           Laplace(0, 1e-4) with exactly floor(n/100) entries, chosen
                  without replacement, multiplied by 100 (outliers): gradients,
                  whose exponents spread wider than weights' and activations'
  normal          N(0, 1)
"""
from __future__ import annotations

import numpy as np

DISTRIBUTIONS = ("half_normal", "weights", "grads", "normal")


def _rng(seed: int) -> np.random.Generator:
    return np.random.default_rng(seed)


def draw(dist: str, shape, seed: int) -> np.ndarray:
    """One float32 array of ``shape`` from distribution ``dist`` under ``seed``."""
    shape = tuple(int(s) for s in (shape if isinstance(shape, (tuple, list)) else (shape,)))
    n = int(np.prod(shape)) if shape else 1
    rng = _rng(seed)
    if dist == "normal":
        x = rng.standard_normal(n)
    elif dist == "half_normal":
        x = np.abs(rng.standard_normal(n))
    elif dist == "weights":
        x = rng.standard_normal(n) * 0.02
    elif dist == "grads":
        x = rng.laplace(0.0, 1e-4, n)
        k = n // 100
        if k:
            idx = rng.choice(n, size=k, replace=False)
            x[idx] *= 100.0
    else:
        raise ValueError("unknown distribution %r" % dist)
    return x.astype(np.float32).reshape(shape)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest even) and widen back."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (b + 0x7FFF + ((b >> 16) & 1)) >> 16 << 16
    return (rounded & 0xFFFFFFFF).astype(np.uint32).view(np.float32).reshape(x.shape)


def gemm_pair_normal(M: int, N: int, K: int, seed: int = 0):
    """A [M, K] then B [K, N] drawn in that order from one N(0,1) stream."""
    rng = _rng(seed)
    a = rng.standard_normal((M, K)).astype(np.float32)
    b = rng.standard_normal((K, N)).astype(np.float32)
    return a, b


def special_values(n: int, seed: int) -> np.ndarray:
    """float32 values that exercise conversion edge cases: zeros of both signs,
    subnormals, powers of two, values just below powers of two, exact ties at
    several LSB scales, the largest finite values and ordinary draws."""
    rng = _rng(seed)
    pool = [0.0, -0.0, 1.0, -1.0, 2.0, 0.5, 1.5, 0.75, 0.375, 3.0, 7.0, 15.0, 0.9999999, 1.9999999,
            np.float32(1.4e-45), np.float32(1e-40), np.float32(-1e-39), np.float32(1.17549435e-38),
            np.float32(3.4028235e38), np.float32(-3.4028235e38), np.float32(1e30), np.float32(1e-30),
            0.25 + 2 ** -10, 1.0 + 2 ** -9, 1.0 + 2 ** -23, 2.0 - 2 ** -22]
    x = rng.standard_normal(n) * np.exp2(rng.integers(-30, 30, n))
    sel = rng.random(n) < 0.5
    x[sel] = rng.choice(np.array(pool, dtype=np.float64), size=int(sel.sum()))
    return x.astype(np.float32)
