"""Reference exploration sampler (test infrastructure only).

The exploration phase of the combined approach (Section 2.3, step 1) measures
the first N schedules that Ansor produces.  Ansor draws initial annotations from
per-rule probability distributions (Section 2.1, "The Initialization of
Annotations"); that figure is missing from the paper, so the reading here is
the uniform distribution over each axis, drawn without replacement over valid
points:

1. Each draw picks an index on every axis in axis order.  The index on an axis
   with n values is ``z mod n`` for the next SplitMix64 output z, redrawn while
   ``z >= floor(2**64 / n) * n`` so that every index is equally likely.
2. A drawn point that is invalid or was already drawn is rejected.
3. Sampling stops after ``n_explore`` distinct valid points or after
   ``100 * n_explore`` drawn points, whichever comes first.

SplitMix64 is re-implemented here from its published definition (Steele, Lea
and Flood, OOPSLA 2014) on Python integers; it shares no code with the library
or with ``synthdata``.

Pins (tests/test_oracle_sampler.py): the published SplitMix64 sequence for
seed 1234567, determinism, no duplicates, ``min(n, |valid|)`` points, and a
chi-square uniformity test on a small lattice.
"""
from __future__ import annotations

MASK = (1 << 64) - 1


class SplitMix64:
    def __init__(self, seed):
        self.state = seed & MASK

    def next(self):
        self.state = (self.state + 0x9E3779B97F4A7C15) & MASK
        z = self.state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK
        return z ^ (z >> 31)

    def below(self, n):
        lim = ((1 << 64) // n) * n
        while True:
            z = self.next()
            if z < lim:
                return z % n


def sample(space, seed, n_explore):
    """Distinct valid points in draw order."""
    rng = SplitMix64(seed)
    seen = set()
    out = []
    draws = 0
    while len(out) < n_explore and draws < 100 * n_explore:
        draws += 1
        idx = tuple(rng.below(n) for n in space.sizes)
        if idx in seen or not space.valid(idx):
            continue
        seen.add(idx)
        out.append(idx)
    return out
