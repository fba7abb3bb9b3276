"""Counter-based SplitMix64 generator for the synthetic workloads.

SplitMix64 (Steele, Lea, Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014) is used as a pure function of a 64-bit counter:
``out(key, i) = mix(key + (i + 1) * GOLDEN)``.  Every tensor gets its own
key, derived from (config name, seed, tensor index), so a tensor's values do
not depend on how many other tensors were drawn before it.

Uniforms take the top 24 bits of ``out`` (exact in fp32); normals come from
the Box-Muller transform of two uniforms, evaluated in float64 and rounded
once to float32.  This module holds no part of the scheduling or operator
arithmetic: it only draws numbers.
"""
from __future__ import annotations

import numpy as np

GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def _mix(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def key_of(*parts) -> np.uint64:
    """Fold ints / strings into one 64-bit stream key."""
    k = np.uint64(0x1234_5678_9ABC_DEF0)
    for p in parts:
        if isinstance(p, str):
            v = 0
            for ch in p.encode():
                v = (v * 131 + ch) & 0xFFFF_FFFF_FFFF_FFFF
            p = v
        with np.errstate(over="ignore"):
            k = _mix(np.uint64(k) ^ np.uint64(int(p) & 0xFFFF_FFFF_FFFF_FFFF))
    return np.uint64(k)


def raw(key: np.uint64, n: int) -> np.ndarray:
    i = np.arange(1, n + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        return _mix(np.uint64(key) + i * GOLDEN)


def uniform01(key: np.uint64, n: int) -> np.ndarray:
    """n values j / 2**24 with j uniform in [0, 2**24), as float64."""
    return (raw(key, n) >> np.uint64(40)).astype(np.float64) * (1.0 / (1 << 24))


def uniform_pm1(key: np.uint64, shape) -> np.ndarray:
    """U(-1, 1) as float32 (exactly representable)."""
    n = int(np.prod(shape)) if len(shape) else 1
    return (2.0 * uniform01(key, n) - 1.0).astype(np.float32).reshape(shape)


def normal(key: np.uint64, shape, std: float) -> np.ndarray:
    """N(0, std^2) as float32 via Box-Muller."""
    n = int(np.prod(shape)) if len(shape) else 1
    m = (n + 1) // 2
    u = uniform01(key, 2 * m)
    u1 = u[0::2] + (1.0 / (1 << 24))       # (0, 1]
    u2 = u[1::2]
    r = np.sqrt(-2.0 * np.log(u1))
    z = np.empty(2 * m, dtype=np.float64)
    z[0::2] = r * np.cos(2.0 * np.pi * u2)
    z[1::2] = r * np.sin(2.0 * np.pi * u2)
    return (z[:n] * std).astype(np.float32).reshape(shape)


class Stream:
    """Sequential draws of small integers / probabilities from one key."""

    def __init__(self, key: np.uint64):
        self.key = np.uint64(key)
        self.i = 0

    def u01(self) -> float:
        self.i += 1
        v = int(raw(self.key + np.uint64(self.i * 7919), 1)[0] >> np.uint64(11))
        return v * (1.0 / (1 << 53))

    def randint(self, n: int) -> int:
        """Uniform integer in [0, n)."""
        return min(int(self.u01() * n), n - 1)
