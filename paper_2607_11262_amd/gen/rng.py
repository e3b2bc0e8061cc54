"""SplitMix64 streams for seeded synthetic inputs.

SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014): the state advances by the golden-ratio increment
0x9E3779B97F4A7C15 and each output is the state passed through the Mix13
finaliser.  Bounded integers use Lemire's multiply-shift reduction
((x * range) >> 64).  Only inputs are drawn here; nothing of the simulation
method lives in this module.
"""
from __future__ import annotations

import math

import numpy as np

_GOLDEN = 0x9E3779B97F4A7C15
_M64 = (1 << 64) - 1


def _mix(z: int) -> int:
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _M64
    return z ^ (z >> 31)


class SplitMix64:
    """A SplitMix64 stream.  ``SplitMix64(seed, stream)`` derives independent
    sub-streams of one seed (stream ids are mixed into the start state)."""

    def __init__(self, seed: int, stream: int = 0):
        self.state = _mix((seed * _GOLDEN + stream) & _M64) if stream else seed & _M64

    def next_u64(self) -> int:
        self.state = (self.state + _GOLDEN) & _M64
        return _mix(self.state)

    def randint(self, lo: int, hi: int) -> int:
        """Uniform integer in the closed range [lo, hi]."""
        span = hi - lo + 1
        assert span >= 1
        return lo + ((self.next_u64() * span) >> 64)

    def choice(self, seq):
        return seq[self.randint(0, len(seq) - 1)]

    def loguniform_int(self, lo: int, hi: int) -> int:
        """Integer whose logarithm is uniform on [ln lo, ln hi] (53-bit draw)."""
        u = (self.next_u64() >> 11) / float(1 << 53)
        return int(math.floor(math.exp(math.log(lo) + u * (math.log(hi) - math.log(lo)))))

    def u64_array(self, n: int) -> np.ndarray:
        return np.array([self.next_u64() for _ in range(n)], dtype=np.uint64)
