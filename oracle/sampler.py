"""Reference exploration sampler (test infrastructure only).

The exploration phase of the combined approach (Section 2.3, step 1) measures
the first N schedules that Ansor produces.  Ansor builds that initial
population by annotating its sketches (Section 2.1, "Sketch annotation" and
"The Initialization of Annotations"); the figure with the per-rule
distributions is missing from the paper, so the reading here is: a sketch is
chosen uniformly, then an annotation uniformly among the sketch's valid ones,
without replacement.  The kernel family (the ``mfma`` knob of the conv and
matmul spaces) stands for the sketch; a generic lattice is one sketch.

1. The valid points of each family are listed in key order.
2. Each draw takes index ``below(F)`` among the F families that still have an
   undrawn valid point (in family order), then index ``below(M)`` among that
   family's M undrawn points, and removes the point.  ``below(n)`` is
   ``z mod n`` for the next SplitMix64 output z, redrawn while
   ``z >= floor(2**64 / n) * n`` so that every index is equally likely.
3. Sampling stops after ``n_explore`` points or when every valid point has
   been drawn.

SplitMix64 is re-implemented here from its published definition (Steele, Lea
and Flood, OOPSLA 2014) on Python integers; it shares no code with the library
or with ``synthdata``.

Pins (tests/test_oracle_sampler.py): the published SplitMix64 sequence for
seed 1234567, determinism, no duplicates, ``min(n, |valid|)`` points, and
chi-square tests that the family of a first draw is uniform over the families
with a valid point and that the point is uniform within its family.
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


def sketch_axis(space):
    """Axis of the kernel-family knob of a conv or matmul space; None for a
    generic lattice."""
    return space.names.index("mfma") if hasattr(space, "op") else None


class Stream:
    """The draw sequence of one space and seed, taken incrementally."""

    def __init__(self, space, seed):
        axis = sketch_axis(space)
        families = {}
        for p in space.valid_points():               # key order
            families.setdefault(0 if axis is None else p[axis], []).append(p)
        self.pools = [families[f] for f in sorted(families)]
        self.rng = SplitMix64(seed)

    def next(self):
        """The next point, or None once every valid point has been drawn."""
        live = [pool for pool in self.pools if pool]
        if not live:
            return None
        pool = live[self.rng.below(len(live))]
        return pool.pop(self.rng.below(len(pool)))


def sample(space, seed, n_explore):
    """Distinct valid points in draw order."""
    out = []
    if n_explore <= 0:
        return out
    stream = Stream(space, seed)
    while len(out) < n_explore:
        p = stream.next()
        if p is None:
            break
        out.append(p)
    return out
