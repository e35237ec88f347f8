"""Counter-based synthetic gradient values (numpy implementation).

The value of element `i` of rank `r` is a pure function of (key = seed + r, i), so any
element can be regenerated on demand without materialising whole tensors, and the
GPU generator in ``workloads/csrc/fill.hip`` produces the same bits from the same
definition.  This module holds no part of the allreduce method.

Definition
----------
* SplitMix64 (Steele, Lea & Flood, "Fast Splittable Pseudorandom Number Generators",
  OOPSLA 2014; 64-bit finaliser constants as published in Vigna's ``splitmix64.c``):
  ``mix(z) = z3`` with ``z1 = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9``,
  ``z2 = (z1 ^ (z1 >> 27)) * 0x94D049BB133111EB``, ``z3 = z2 ^ (z2 >> 31)``, all mod 2^64.
  The n-th output (n = 0, 1, ...) of a generator seeded with S is ``mix(S + (n+1)*G)``
  with the golden-ratio increment ``G = 0x9E3779B97F4A7C15``.
* Each key owns the stream seeded with ``S = mix(key + G)``; element ``i`` uses the
  stream outputs ``4i, 4i+1, 4i+2, 4i+3``.
* ``uniform``: the top 24 bits ``k`` of output ``4i`` give ``(2k + 1 - 2^24) * 2^-24``,
  a midpoint of one of 2^24 equal cells of (-1, 1), exact in binary32.
* ``normal`` (mean 0, standard deviation sigma): the Irwin-Hall approximation with twelve
  uniforms, ``sum(U_1..U_12) - 6``, whose variance is exactly 1.  The twelve uniforms are
  the 21-bit fields at bit offsets 0, 21 and 42 of outputs ``4i .. 4i+3``, taken as cell
  midpoints ``(k + 1/2) * 2^-21``.  With ``K`` the sum of the twelve integers the value is
  ``z = (K + 6 - 6 * 2^21) * 2^-21``; the numerator is an integer below 2^24 in magnitude,
  so ``z`` is exact in binary32, and the result is the binary32 product ``z * sigma32``
  (one round-to-nearest-even), with ``sigma32`` the binary32 value nearest sigma.
  Only integer operations and one correctly rounded multiply are involved, so CPU and
  GPU agree bit for bit.
"""
from __future__ import annotations

import numpy as np

__all__ = ["GAMMA", "mix", "stream_seed", "draw", "uniform", "normal", "values"]

GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
_MASK21 = np.uint64((1 << 21) - 1)


def mix(z):
    """SplitMix64 finaliser on a uint64 array (wrap-around arithmetic)."""
    z = np.asarray(z, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def stream_seed(key: int) -> np.uint64:
    with np.errstate(over="ignore"):
        return mix(np.array([key], dtype=np.uint64) + GAMMA)[0]


def draw(key: int, idx, j: int):
    """Stream output ``4*idx + j`` for the stream of `key` (uint64 array)."""
    s = stream_seed(key)
    idx = np.asarray(idx, dtype=np.uint64)
    with np.errstate(over="ignore"):
        n = idx * np.uint64(4) + np.uint64(j + 1)
        return mix(s + n * GAMMA)


def uniform(key: int, idx) -> np.ndarray:
    """Values in (-1, 1) at element indices `idx` (binary32)."""
    k = (draw(key, idx, 0) >> np.uint64(40)).astype(np.int64)
    num = 2 * k + 1 - (1 << 24)  # |num| < 2^24: exact in binary32
    return (num.astype(np.float32) * np.float32(2.0 ** -24)).astype(np.float32)


def normal(key: int, idx, sigma: float = 0.01) -> np.ndarray:
    """Irwin-Hall(12) normal values with standard deviation `sigma` (binary32)."""
    idx = np.asarray(idx, dtype=np.uint64)
    total = np.zeros(idx.shape, dtype=np.int64)
    for j in range(4):
        d = draw(key, idx, j)
        for shift in (0, 21, 42):
            total += ((d >> np.uint64(shift)) & _MASK21).astype(np.int64)
    num = total + 6 - 6 * (1 << 21)  # |num| <= 6 * 2^21 < 2^24
    z = num.astype(np.float32) * np.float32(2.0 ** -21)  # exact
    return (z * np.float32(sigma)).astype(np.float32)


def values(dist: str, key: int, idx, sigma: float = 0.01) -> np.ndarray:
    if dist == "uniform":
        return uniform(key, idx)
    if dist == "normal":
        return normal(key, idx, sigma)
    raise ValueError(f"unknown distribution {dist!r}")
