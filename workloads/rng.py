"""Counter-based random numbers for the seeded synthetic workloads.

Every draw is a pure function of (seed, stream name, index), so the same
workload comes out on any machine and in any order of generation.

``mix`` is the output function of SplitMix64 (Steele, Lea and Flood,
"Fast splittable pseudorandom number generators", OOPSLA 2014) applied to
the state ``x``: add the golden-ratio increment, then two xor-shift-multiply
rounds and a final xor-shift.  ``stream_key`` names a stream by the 64-bit
FNV-1a hash of its name.

This module draws input data only (lags, byte counts, permutations,
degraded cables).  It holds none of the simulator's arithmetic.
"""

from __future__ import annotations

import numpy as np

MASK64 = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15
M1 = 0xBF58476D1CE4E5B9
M2 = 0x94D049BB133111EB


def mix(x: int) -> int:
    """SplitMix64 output for state ``x`` (scalar, Python ints)."""
    z = (x + GOLDEN) & MASK64
    z = ((z ^ (z >> 30)) * M1) & MASK64
    z = ((z ^ (z >> 27)) * M2) & MASK64
    return z ^ (z >> 31)


def mix_np(x: np.ndarray) -> np.ndarray:
    """Vectorised ``mix`` over a uint64 array (numpy wraps modulo 2**64)."""
    with np.errstate(over="ignore"):
        z = x.astype(np.uint64) + np.uint64(GOLDEN)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(M1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(M2)
        return z ^ (z >> np.uint64(31))


def fnv1a64(name: str) -> int:
    h = 0xCBF29CE484222325
    for b in name.encode():
        h ^= b
        h = (h * 0x100000001B3) & MASK64
    return h


def stream_key(seed: int, name: str) -> int:
    return mix(mix(seed & MASK64) ^ fnv1a64(name))


class Stream:
    """Named stream of 64-bit draws: draw i is ``mix(key + i)``."""

    def __init__(self, seed: int, name: str):
        self.key = stream_key(seed, name)

    def u64(self, n: int, start: int = 0) -> np.ndarray:
        idx = np.arange(start, start + n, dtype=np.uint64)
        with np.errstate(over="ignore"):
            return mix_np(np.uint64(self.key) + idx)

    def u01(self, n: int, start: int = 0) -> np.ndarray:
        """Uniform doubles in [0, 1): the top 53 bits times 2**-53."""
        return (self.u64(n, start) >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)

    def below(self, bound: int, n: int, start: int = 0) -> np.ndarray:
        """Integers in [0, bound): floor(u01 * bound) (bias < 2**-40 here)."""
        return np.minimum((self.u01(n, start) * bound).astype(np.int64), bound - 1)

    def permutation(self, n: int, start: int = 0) -> np.ndarray:
        """Fisher-Yates shuffle of 0..n-1 driven by draws start..start+n-2."""
        p = np.arange(n, dtype=np.int64)
        if n <= 1:
            return p
        u = self.u01(n - 1, start)
        for i in range(n - 1, 0, -1):
            j = min(int(u[n - 1 - i] * (i + 1)), i)
            p[i], p[j] = p[j], p[i]
        return p

    def sample_without_replacement(self, n: int, k: int, start: int = 0) -> np.ndarray:
        """First k entries of a partial Fisher-Yates shuffle of 0..n-1."""
        p = np.arange(n, dtype=np.int64)
        u = self.u01(k, start)
        for i in range(k):
            j = i + min(int(u[i] * (n - i)), n - i - 1)
            p[i], p[j] = p[j], p[i]
        return p[:k].copy()
