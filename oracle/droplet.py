"""Reference Droplet Search and combined explore/exploit driver (test infrastructure only).

Droplet Search (Section 2.2) is coordinate descent over the annotation
lattice of one sketch:

1. At iteration zero the current candidate is the point that applies no
   optimisation (or, in the combined approach of Section 2.3, the best of the
   N explored schedules).
2. While some point that differs from the current one in a single coordinate
   (a neighbour, Example 3) yields a faster kernel, move there; when none
   does, stop.

Readings taken where the paper is silent or loose:

* Step 2 admits first- or best-improvement; the move taken here is to the
  fastest neighbour (ties go to the first neighbour in neighbour order).
* "Faster" is statistical (Section 3, RQ4 and RQ5: the search stops when the
  neighbours are not significantly different at 95% confidence).  The test
  used is the one-sided Wilcoxon rank-sum (Mann-Whitney U) test on the
  per-repeat times, normal approximation with tie and continuity correction,
  the test family the paper uses for its own reporting (Section 3,
  "Confidence").  A move needs a lower median *and* p < alpha (0.05).  With
  ``alpha >= 1`` the comparison is the plain strict ``median < median``
  (used with deterministic costs).
* Droplet runs at most 100 trials (Section 3, RQ2).  ``budget`` caps the new
  neighbour measurements; the start point, when not already measured, is
  measured once more and reported in ``measured`` but not charged to the
  budget.  Measured points are cached and never measured twice; a failed
  measurement has infinite time and still counts.  When the budget runs out
  part-way through a neighbourhood, the neighbours already measured in it are
  still compared with the current point (and the move taken if one is
  faster) before the search stops: the paper's stopping rule is the trial
  count, and a trial that was run is part of the search.
* ``frozen`` lists axes that are held at the start's value (the single-sketch
  variant of Section 2.2's first limitation).
* ``line`` (not the method of the paper's experiments): Section 2.2 presents
  Droplet Search without the speculative steps of its original description
  and calls it a line search; the reading taken for those steps is that a move
  along axis a in direction d is followed by further steps along (a, d), each
  a charged trial, for as long as the next point is in range, valid and better
  than the current one.  The neighbourhood scan then resumes from the last
  point reached.

Pins of ``line`` (tests/test_oracle_droplet.py): a trace worked by hand on a
separable 5x5 bowl, exhaustive search on convex costs, fewer trials than the
plain search on long one-axis descents.

Pins (tests/test_oracle_droplet.py): a trace worked by hand on the lattice of
Example 3 (tests/golden/droplet_trace_example3.txt), exhaustive search on small
lattices with convex costs, local optimality and budget invariants, and the
p-value against ``scipy.stats.mannwhitneyu``.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

from . import sampler as _sampler

OK = 0
EBUDGET = -6
EEXHAUSTED = -7


@dataclass
class Meas:
    median: float
    repeats: list = field(default_factory=list)
    status: int = 0

    @staticmethod
    def of(value):
        if isinstance(value, Meas):
            return value
        if isinstance(value, (list, tuple)):
            r = [float(t) for t in value]
            return Meas(_median(r), r, 0)
        v = float(value)
        return Meas(v, [v], 0 if math.isfinite(v) else -5)


def _median(r):
    s = sorted(r)
    n = len(s)
    if n == 0:
        return math.inf
    return s[n // 2] if n % 2 else 0.5 * (s[n // 2 - 1] + s[n // 2])


def ranksum_p_less(a, b):
    """One-sided p-value that sample ``a`` is stochastically smaller than ``b``."""
    n1, n2 = len(a), len(b)
    if n1 == 0 or n2 == 0:
        return 1.0
    pooled = sorted([(v, 0) for v in a] + [(v, 1) for v in b])
    n = n1 + n2
    ranks = [0.0] * n
    ties = 0.0
    i = 0
    while i < n:
        j = i
        while j + 1 < n and pooled[j + 1][0] == pooled[i][0]:
            j += 1
        r = 0.5 * (i + j) + 1.0          # average of ranks i+1 .. j+1
        for t in range(i, j + 1):
            ranks[t] = r
        g = j - i + 1
        ties += g ** 3 - g
        i = j + 1
    r1 = sum(ranks[t] for t in range(n) if pooled[t][1] == 0)
    u1 = r1 - n1 * (n1 + 1) / 2.0
    mu = n1 * n2 / 2.0
    var = n1 * n2 / 12.0 * ((n + 1) - ties / (n * (n - 1)))
    if var <= 0.0:
        return 1.0
    z = (u1 - mu + 0.5) / math.sqrt(var)
    return 0.5 * math.erfc(-z / math.sqrt(2.0))


def better(a: Meas, b: Meas, alpha: float) -> bool:
    if a.status != 0 or not math.isfinite(a.median):
        return False
    if b.status != 0 or not math.isfinite(b.median):
        return True
    if not a.median < b.median:
        return False
    if alpha >= 1.0:
        return True
    return ranksum_p_less(a.repeats, b.repeats) < alpha


def droplet(space, cost, start=None, budget=100, alpha=1.0, cache=None, frozen=(), line=False):
    """Returns dict(best, meas, measured, status, path, order).

    ``cost(idx)`` returns a float, a list of repeat times, or a Meas.
    ``cache`` maps key -> Meas and is updated in place when given.
    """
    cache = {} if cache is None else cache
    order = []                      # keys measured by this call, in order
    cur = space.origin() if start is None else tuple(start)
    if cur is None:
        return dict(best=None, meas=None, measured=0, status=EEXHAUSTED, path=[], order=order)
    start_measured = 0              # 1 if the start had to be measured here
    nb_measured = 0                 # neighbour measurements, charged to the budget
    k = space.key(cur)
    if k not in cache:
        cache[k] = Meas.of(cost(cur))
        start_measured = 1
        order.append(k)
    path = [cur]
    status = OK
    while True:
        nbs = [nb for nb in space.neighbors(cur)
               if all(nb[a] == cur[a] for a in frozen)]
        stop = False
        for nb in nbs:
            kn = space.key(nb)
            if kn in cache:
                continue
            if nb_measured >= budget:
                status = EBUDGET
                stop = True
                break
            cache[kn] = Meas.of(cost(nb))
            nb_measured += 1
            order.append(kn)
        # The fastest neighbour among those measured (ties: first in neighbour
        # order).  A budget stop part-way through the neighbourhood still lets
        # the neighbours measured before it compete: their trials were spent.
        best_nb = None
        for nb in nbs:
            if space.key(nb) not in cache:
                continue
            if best_nb is None or cache[space.key(nb)].median < cache[space.key(best_nb)].median:
                best_nb = nb
        if best_nb is None:
            break
        if not better(cache[space.key(best_nb)], cache[space.key(cur)], alpha):
            break
        axis = next(a for a in range(len(cur)) if best_nb[a] != cur[a])
        step = best_nb[axis] - cur[axis]
        cur = best_nb
        path.append(cur)
        while line:
            nxt = list(cur)
            nxt[axis] += step
            nxt = tuple(nxt)
            if not 0 <= nxt[axis] < space.sizes[axis] or not space.valid(nxt):
                break
            kn = space.key(nxt)
            if kn not in cache:
                if nb_measured >= budget:
                    status = EBUDGET
                    stop = True
                    break
                cache[kn] = Meas.of(cost(nxt))
                nb_measured += 1
                order.append(kn)
            if not better(cache[kn], cache[space.key(cur)], alpha):
                break
            cur = nxt
            path.append(cur)
        if stop:
            break
    return dict(best=cur, meas=cache[space.key(cur)], measured=start_measured + nb_measured,
                status=status, path=path, order=order)


def combined(space, cost, seed, n_explore=300, budget=100, alpha=1.0, frozen=()):
    """Section 2.3: explore ``n_explore`` sampled schedules, hand the best to
    Droplet Search, run it to convergence (or the budget)."""
    pts = _sampler.sample(space, seed, n_explore)
    if not pts:
        return dict(best=None, status=EEXHAUSTED, n_explore=0, n_droplet=0)
    cache = {}
    best, best_m = None, None
    for p in pts:
        m = Meas.of(cost(p))
        cache[space.key(p)] = m
        if best is None or m.median < best_m.median:
            best, best_m = p, m
    d = droplet(space, cost, start=best, budget=budget, alpha=alpha, cache=cache, frozen=frozen)
    return dict(best=d["best"], meas=d["meas"], status=d["status"], n_explore=len(pts),
                n_droplet=d["measured"], seed_point=best, path=d["path"], samples=pts)
