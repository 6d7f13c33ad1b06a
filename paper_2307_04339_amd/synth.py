"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle checks.

This module holds only random-number draws and storage-format conversions
(rounding a float64 draw to fp32/fp16/bf16 bits).  It contains none of the
operators' arithmetic, so both the HIP path and the CPU oracle can be fed from
it without sharing any computation.

All draws use ``numpy.random.default_rng`` with explicit seeds; a per-tensor
seed is derived from (config seed, layer index, tensor name) with CRC32 so the
same tensor is reproduced in any process.
"""
from __future__ import annotations

import zlib

import numpy as np

DTYPES = ("f32", "f16", "bf16")


def tensor_seed(seed: int, layer: int, name: str) -> int:
    """Stable per-tensor seed."""
    return (zlib.crc32(f"{seed}:{layer}:{name}".encode()) ^ (seed * 0x9E3779B1)) & 0xFFFFFFFF


def uniform(shape, lo=-1.0, hi=1.0, seed=0) -> np.ndarray:
    """float64 draw from U[lo, hi)."""
    rng = np.random.default_rng(seed)
    return rng.uniform(lo, hi, size=shape)


def integers(shape, lo, hi, seed=0) -> np.ndarray:
    """float64 array of integers in [lo, hi] (exact in every storage type for small values)."""
    rng = np.random.default_rng(seed)
    return rng.integers(lo, hi + 1, size=shape).astype(np.float64)


def bf16_bits(x64: np.ndarray) -> np.ndarray:
    """Round float64 values to bfloat16 (round to nearest even) and return the uint16 bits."""
    f = np.ascontiguousarray(x64, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    u = (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16)
    return u.view(np.float32).astype(np.float64)


def to_storage(x64: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 values to the storage dtype; returns an array whose raw bytes
    are the device representation (float32, float16, or uint16 for bf16)."""
    if dtype == "f32":
        return np.ascontiguousarray(x64, dtype=np.float32)
    if dtype == "f16":
        return np.ascontiguousarray(x64, dtype=np.float16)
    if dtype == "bf16":
        return bf16_bits(x64)
    raise ValueError(dtype)


def storage_to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of stored values to float64."""
    if dtype == "bf16":
        return bf16_to_f64(a)
    return np.asarray(a, dtype=np.float64)


def storage_tensor(shape, dtype, seed, lo=-1.0, hi=1.0):
    """(storage array, exact float64 view) for a U[lo,hi) tensor."""
    s = to_storage(uniform(shape, lo, hi, seed), dtype)
    return s, storage_to_f64(s, dtype)


# ------------------------------------------------------------- arrivals
def periodic_releases(n: int, period_ns: int, start_ns: int = 0) -> np.ndarray:
    """Uniform arrivals: one release every period."""
    return start_ns + period_ns * np.arange(n, dtype=np.int64)


def poisson_releases(n: int, mean_ns: float, seed: int, start_ns: int = 0) -> np.ndarray:
    """Poisson arrivals: exponential inter-arrival gaps with the given mean."""
    rng = np.random.default_rng(seed)
    gaps = rng.exponential(mean_ns, size=n)
    gaps[0] = 0.0
    return start_ns + np.cumsum(gaps).astype(np.int64)
