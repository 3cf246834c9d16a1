"""Counter-based splitmix64 random streams for the synthetic workloads.

Every value is a pure function of (seed, stream name, counter), so the same
seed always yields the same bytes on any machine.  The mixing function is the
published splitmix64 finaliser (Steele, Lea and Flood, "Fast splittable
pseudorandom number generators", OOPSLA 2014).

This module holds random-number plumbing only: nothing of the lattice method.
"""
from __future__ import annotations

import zlib

import numpy as np

_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def _mix(z: np.ndarray) -> np.ndarray:
    """splitmix64 output function applied elementwise to uint64 states."""
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        return z ^ (z >> np.uint64(31))


class Stream:
    """One named random stream: draws consume consecutive counters."""

    def __init__(self, seed: int, name: str):
        tag = zlib.crc32(name.encode()) & 0xFFFFFFFF
        base = np.array([(int(seed) & 0xFFFFFFFF) << 32 | tag], dtype=np.uint64)
        self._base = _mix(base)[0]
        self._ctr = 0

    def bits(self, n: int) -> np.ndarray:
        """n raw uint64 draws."""
        idx = np.arange(self._ctr + 1, self._ctr + 1 + n, dtype=np.uint64)
        self._ctr += n
        with np.errstate(over="ignore"):
            return _mix(self._base + idx * _GAMMA)

    def uniform(self, n: int) -> np.ndarray:
        """n doubles in [0, 1): top 24 bits times 2^-24 (exact in fp32 too)."""
        return (self.bits(n) >> np.uint64(40)).astype(np.float64) * (2.0 ** -24)

    def uniform_range(self, n: int, lo: float, hi: float) -> np.ndarray:
        return lo + (hi - lo) * self.uniform(n)

    def normal(self, n: int) -> np.ndarray:
        """n standard normal doubles by the Box-Muller transform."""
        k = (n + 1) // 2
        u1 = 1.0 - self.uniform(k)          # (0, 1]
        u2 = self.uniform(k)
        r = np.sqrt(-2.0 * np.log(u1))
        z = np.concatenate([r * np.cos(2.0 * np.pi * u2), r * np.sin(2.0 * np.pi * u2)])
        return z[:n]

    def integers(self, n: int, lo: int, hi: int) -> np.ndarray:
        """n integers uniform in [lo, hi) (hi - lo < 2^24)."""
        span = hi - lo
        return lo + np.minimum((self.uniform(n) * span).astype(np.int64), span - 1)

    def permutation(self, n: int) -> np.ndarray:
        """A uniformly random permutation of range(n) (sort of random keys)."""
        return np.argsort(self.bits(n), kind="stable")
