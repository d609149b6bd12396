"""Integer random streams used by clustering and sampling.

The paper does not fix a generator.  The reading used here:
  * SplitMix64 (Steele, Lea and Flood, 2014): state += 0x9E3779B97F4A7C15,
    output = mix64(state), where mix64 is its finaliser.
  * Bounded integers in [0, r) by Lemire's multiply-shift with rejection
    ("Fast Random Integer Generation in an Interval", 2019).
  * Derived keys: a chain of mix64 over (seed + tag, a, b, ...), with every
    addition taken modulo 2^64.
All arithmetic is on Python integers masked to 64 bits.
"""
from __future__ import annotations

MASK64 = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15
TAG_ASSIGN = 0x41535349474E  # "ASSIGN"
TAG_SAMPLE = 0x53414D504C45  # "SAMPLE"


def mix64(z: int) -> int:
    """SplitMix64 output finaliser."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


class SplitMix64:
    """The SplitMix64 stream: each draw advances the state by the golden gamma."""

    def __init__(self, state: int):
        self.state = state & MASK64

    def next(self) -> int:
        self.state = (self.state + GOLDEN) & MASK64
        return mix64(self.state)


def bounded(gen: SplitMix64, r: int) -> int:
    """Uniform integer in [0, r): keep the high word of x*r, reject the biased
    low words (those below 2^64 mod r)."""
    assert 0 < r <= MASK64
    m = gen.next() * r
    low = m & MASK64
    if low < r:
        threshold = ((1 << 64) - r) % r
        while low < threshold:
            m = gen.next() * r
            low = m & MASK64
    return m >> 64


def derive_key(seed: int, tag: int, *parts: int) -> int:
    """key = mix64(...mix64(mix64(seed + tag) + parts[0]) + parts[1]...)."""
    h = mix64((seed + tag) & MASK64)
    for p in parts:
        h = mix64((h + p) & MASK64)
    return h
