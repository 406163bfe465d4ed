"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle checks.

This module only draws random numbers and casts them to the storage dtypes; it holds
none of the layer's arithmetic. Every tensor comes from its own PCG64 stream, keyed
by (seed, tensor name), so a tensor does not depend on which other tensors were
drawn. Activations are drawn at the largest row count and sliced, so the weights and
the first rows of X are identical across M.

Distributions stand in for trained LLaMA-2 layers and C4/WikiText activations, which
are not available here:

* W fp32 ~ N(0, 0.02^2)
* X ~ N(0, 1), cast to bf16 or fp16 with round-to-nearest-even
* L, R fp16 ~ N(0, 0.01^2)
* outlier variant: floor(0.01 K) input channels, chosen without replacement,
  scaled by 20 before the cast (activation outliers discussed in the SLiM chapter)
"""
from __future__ import annotations

import zlib

import numpy as np


def stream(seed: int, name: str) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed), zlib.crc32(name.encode())])))


def bf16_bits(x32: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round to nearest even (finite inputs)."""
    b = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f16_to_f64(bits: np.ndarray) -> np.ndarray:
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def weights(n: int, k: int, seed: int = 0, name: str = "W", std: float = 0.02) -> np.ndarray:
    """fp32 [n, k] ~ N(0, std^2)."""
    return (stream(seed, name).standard_normal((n, k), dtype=np.float32) * np.float32(std)).astype(np.float32)


def activations(m: int, k: int, seed: int = 0, name: str = "X", dtype: str = "bf16",
                outliers: bool = False, scale: float = 1.0) -> tuple[np.ndarray, np.ndarray]:
    """Returns (bits uint16 [m, k], values float64 [m, k]) for dtype 'bf16' or 'fp16'.

    ``scale`` multiplies the N(0, 1) draws (in float32) before the cast: gradient-sized inputs
    (1e-3 .. 1e-7) or activations beyond the fp16 range (1e6 in bf16)."""
    x = stream(seed, name).standard_normal((m, k), dtype=np.float32)
    if outliers:
        ch = stream(seed, name + "/outlier_channels").choice(k, size=int(0.01 * k), replace=False)
        x[:, ch] *= np.float32(20.0)
    if scale != 1.0:
        x *= np.float32(scale)
    if dtype == "bf16":
        bits = bf16_bits(x)
        return bits, bf16_to_f64(bits)
    if dtype == "fp16":
        h = x.astype(np.float16)
        return h.view(np.uint16).copy(), h.astype(np.float64)
    raise ValueError(dtype)


def adapter(k: int, n: int, r: int, seed: int = 0, name: str = "", std: float = 0.01):
    """fp16 L [k, r] and R [r, n] ~ N(0, std^2); returns bit patterns (uint16) and float64 values."""
    L = (stream(seed, name + "L").standard_normal((k, r), dtype=np.float32) * np.float32(std)).astype(np.float16)
    R = (stream(seed, name + "R").standard_normal((r, n), dtype=np.float32) * np.float32(std)).astype(np.float16)
    return (L.view(np.uint16).copy(), R.view(np.uint16).copy(), L.astype(np.float64), R.astype(np.float64))
