"""SplitMix64 for the oracle's scheduler draws -- test infrastructure only.

The group generator draws random numbers (group sizes, members, partitions).
Those draws cannot be passed in as inputs for a stateful generator that runs
for thousands of steps, so each side of the parity check implements the same
published generator on its own.  This is the oracle's copy.

Definition (Steele, Lea & Flood, OOPSLA 2014, 64-bit output function):
  state <- state + 0x9E3779B97F4A7C15
  z <- state; z <- (z ^ z>>30) * 0xBF58476D1CE4E5B9
              z <- (z ^ z>>27) * 0x94D049BB133111EB
  out <- z ^ z>>31                       (all arithmetic mod 2^64)

Keys fold components c_1, c_2, ... into the seed: k <- mix(k + GAMMA*(c+1)).
Bounded draws use the multiply-shift map of Lemire ("Fast random integer
generation in an interval", 2019) without the rejection step:
  bounded(n) = ((x >> 32) * n) >> 32,  0 <= result < n  (n < 2^32).
"""
from __future__ import annotations

GAMMA = 0x9E3779B97F4A7C15
_M = (1 << 64) - 1


def mix(z: int) -> int:
    z &= _M
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _M
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _M
    return z ^ (z >> 31)


def fold(seed: int, *components: int) -> int:
    k = seed & _M
    for c in components:
        k = mix(k + GAMMA * (c + 1))
    return k


class Stream:
    """Sequential SplitMix64 stream."""

    def __init__(self, state: int):
        self.state = state & _M

    def next(self) -> int:
        self.state = (self.state + GAMMA) & _M
        return mix(self.state)

    def bounded(self, n: int) -> int:
        assert 0 < n < (1 << 32)
        return ((self.next() >> 32) * n) >> 32
