"""Seeded synthetic input generators shared by the oracle checks, the GPU tests
and the benchmark.

This module draws random numbers and rounds them to the storage precision of a
workload; it holds none of the method's arithmetic (no convolution, product,
normalisation or save rule).  Every array is produced on the host with numpy's
PCG64 bit generator from an explicit integer seed, so the oracle and the HIP
path always see bit-identical inputs.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "rng", "normal", "uniform", "kaiming_uniform", "round_bf16",
    "cast", "DTYPES",
]

DTYPES = ("f32", "bf16")


def rng(seed: int) -> np.random.Generator:
    """A fresh PCG64 generator for one tensor."""
    return np.random.Generator(np.random.PCG64(int(seed)))


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 value, ties to even.

    Returns float32 values that are exactly representable in bfloat16.
    Inputs here are finite draws; NaN/Inf are passed through unchanged.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    # 32-bit arithmetic: a finite value's bits are at most 0xFF7FFFFF, so
    # adding 0x8000 cannot wrap (only NaN payloads could, and NaN/Inf take
    # the np.where branch)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    out = r.view(np.float32).reshape(a.shape)
    finite = np.isfinite(a)
    return np.where(finite, out, a).astype(np.float32, copy=False)


def cast(a: np.ndarray, dtype: str) -> np.ndarray:
    """Bring float32 draws to the storage precision `dtype` ('f32'|'bf16')."""
    if dtype == "f32":
        return np.ascontiguousarray(a, dtype=np.float32)
    if dtype == "bf16":
        return round_bf16(a)
    raise ValueError(f"unknown dtype {dtype!r}")


def normal(shape, seed: int, std: float = 1.0, mean: float = 0.0,
           dtype: str = "f32") -> np.ndarray:
    g = rng(seed)
    a = g.standard_normal(size=tuple(shape), dtype=np.float32)
    if std != 1.0 or mean != 0.0:
        a = (a * np.float32(std) + np.float32(mean)).astype(np.float32)
    return cast(a, dtype)


def uniform(shape, seed: int, lo: float, hi: float,
            dtype: str = "f32") -> np.ndarray:
    g = rng(seed)
    a = g.uniform(lo, hi, size=tuple(shape)).astype(np.float32)
    return cast(a, dtype)


def kaiming_uniform(shape, seed: int, fan_in: int, dtype: str = "f32") -> np.ndarray:
    """U(-1/sqrt(fan_in), +1/sqrt(fan_in)): the default init bound of a
    PyTorch Conv2d/Linear weight (kaiming-uniform with a = sqrt(5))."""
    bound = 1.0 / float(np.sqrt(fan_in))
    return uniform(shape, seed, -bound, bound, dtype)
