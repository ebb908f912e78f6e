"""Pins of the reference Droplet Search driver."""
import itertools
import math

import numpy as np
import pytest
from scipy import stats

from oracle import droplet as dr
from oracle import space as sp


def example3_lattice():
    return sp.Lattice([[1, 2, 3, 4, 5], [1, 2, 4, 8, 16]], ["unroll", "tile"])


def example3_cost(lat):
    def cost(idx):
        u, t = lat.values[0][idx[0]], lat.values[1][idx[1]]
        return (u - 4) ** 2 + (math.log2(t) - 1) ** 2
    return cost


def test_hand_trace(golden_dir):
    rows = {}
    for line in open(f"{golden_dir}/droplet_trace_example3.txt"):
        if line.strip() and not line.startswith("#"):
            head, *rest = line.split()
            rows[head] = rest
    lat = example3_lattice()
    calls = []
    base = example3_cost(lat)

    def cost(idx):
        calls.append(idx)
        return base(idx)

    res = dr.droplet(lat, cost, start=None, budget=100)
    as_vals = lambda p: f"{lat.values[0][p[0]]},{lat.values[1][p[1]]}"
    assert [as_vals(p) for p in res["path"]] == rows["path"]
    assert [as_vals(p) for p in calls] == rows["order"]
    assert res["measured"] == int(rows["total_measurements"][0])
    assert res["measured"] - 1 == int(rows["neighbor_measurements"][0])
    assert res["meas"].median == float(rows["best_cost"][0]) and res["status"] == dr.OK


def test_budget_stops_and_counts():
    # Worked by hand on Example 3's lattice, cost (u-4)^2 + (log2 t - 1)^2 from
    # (u,t) = (1,1) (cost 10), budget 3.  Scan 1: (2,1) = 5 and (1,2) = 9, two
    # trials; move to (2,1).  Scan 2: (1,1) is cached, (3,1) = 2 is the third
    # trial, (2,2) would be the fourth: the budget stops the scan there, but
    # (3,1) was measured and beats (2,1), so the search ends on it.
    lat = example3_lattice()
    res = dr.droplet(lat, example3_cost(lat), budget=3)
    assert res["status"] == dr.EBUDGET and res["measured"] == 4
    assert [tuple(p) for p in res["path"]] == [(0, 0), (1, 0), (2, 0)]
    assert res["best"] == (2, 0) and res["meas"].median == 2.0
    # budget 2: scan 2 stops before (3,1), nothing measured there beats (2,1)
    res2 = dr.droplet(lat, example3_cost(lat), budget=2)
    assert res2["status"] == dr.EBUDGET and res2["best"] == (1, 0) and res2["measured"] == 3
    res0 = dr.droplet(lat, example3_cost(lat), budget=0)
    assert res0["status"] == dr.EBUDGET and res0["measured"] == 1 and res0["best"] == (0, 0)


def convex_cost(centers, weights):
    def cost(idx):
        return sum(w * (i - c) ** 2 for i, c, w in zip(idx, centers, weights))
    return cost


@pytest.mark.parametrize("seed", range(6))
def test_exhaustive_convex_every_start(seed):
    rng = np.random.default_rng(seed)
    lat = sp.Lattice([list(range(4)), list(range(4)), list(range(3))])
    centers = rng.uniform(0, 3, size=3)
    weights = rng.uniform(0.5, 2.0, size=3) + np.array([0.0, 1e-3, 2e-3]) * math.pi
    cost = convex_cost(centers, weights)
    gmin = min(lat.valid_points(), key=cost)
    for start in lat.valid_points():
        res = dr.droplet(lat, cost, start=start, budget=1000)
        assert res["best"] == gmin


def bowl(p):
    return (p[0] - 4) ** 2 + (p[1] - 4) ** 2


def test_line_hand_trace():
    # Worked by hand on a 5x5 lattice, cost (i-4)^2 + (j-4)^2, start (0,0): the
    # first scan measures (1,0) and (0,1) (both 25) and moves to the first;
    # steps along +i measure (2,0) 20, (3,0) 17, (4,0) 16 and stop at the edge;
    # the scan of (4,0) measures (4,1) 9 and moves; steps along +j measure
    # (4,2) 4, (4,3) 1, (4,4) 0; the scan of (4,4) measures (3,4) 1 and stops.
    lat = sp.Lattice([list(range(5)), list(range(5))])
    calls = []

    def cost(p):
        calls.append(tuple(p))
        return bowl(p)

    res = dr.droplet(lat, cost, start=(0, 0), line=True)
    assert calls == [(0, 0), (1, 0), (0, 1), (2, 0), (3, 0), (4, 0), (4, 1), (4, 2), (4, 3),
                     (4, 4), (3, 4)]
    assert res["path"] == [(0, 0), (1, 0), (2, 0), (3, 0), (4, 0), (4, 1), (4, 2), (4, 3),
                           (4, 4)]
    assert res["measured"] == 11 and res["best"] == (4, 4) and res["status"] == dr.OK
    plain = dr.droplet(lat, bowl, start=(0, 0))
    assert plain["best"] == (4, 4) and plain["measured"] > res["measured"]


def test_line_budget_stops_inside_a_line():
    lat = sp.Lattice([list(range(5)), list(range(5))])
    res = dr.droplet(lat, bowl, start=(0, 0), budget=3, line=True)
    # (1,0) and (0,1) by the scan, (2,0) by the first step; the next step is over budget
    assert res["status"] == dr.EBUDGET and res["measured"] == 4 and res["best"] == (2, 0)


def test_line_stops_at_invalid_points_and_worse_steps():
    # (3,0) is invalid: the line along +i stops at (2,0) without measuring it
    lat = sp.Lattice([list(range(5)), list(range(3))], predicate=lambda p: p != (3, 0))
    calls = []

    def cost(p):
        calls.append(tuple(p))
        return (p[0] - 4) ** 2 + 3 * p[1]

    res = dr.droplet(lat, cost, start=(0, 0), line=True)
    assert (3, 0) not in calls
    # from (2,0) the scan goes to (2,1)... only if better; (2,1) costs 7 > 4, so it stops
    assert res["best"] == (2, 0) and all(lat.valid(p) for p in calls)


@pytest.mark.parametrize("seed", range(6))
def test_line_exhaustive_convex_every_start(seed):
    rng = np.random.default_rng(seed)
    lat = sp.Lattice([list(range(5)), list(range(4)), list(range(3))])
    centers = rng.uniform(0, 4, size=3)
    weights = rng.uniform(0.5, 2.0, size=3) + np.array([0.0, 1e-3, 2e-3]) * math.pi
    cost = convex_cost(centers, weights)
    gmin = min(lat.valid_points(), key=cost)
    for start in lat.valid_points():
        res = dr.droplet(lat, cost, start=start, budget=1000, line=True)
        assert res["best"] == gmin


@pytest.mark.parametrize("seed", range(10))
def test_line_fewer_trials_on_one_axis_descents(seed):
    # long axes, separable convex cost, start in a corner: steps replace scans
    rng = np.random.default_rng(300 + seed)
    lat = sp.Lattice([list(range(12)), list(range(10)), list(range(3))])
    cost = convex_cost(rng.uniform(8, 11, size=3) * [1, 0.9, 0.2], rng.uniform(0.5, 2.0, size=3))
    a = dr.droplet(lat, cost, start=(0, 0, 0), budget=1000)
    b = dr.droplet(lat, cost, start=(0, 0, 0), budget=1000, line=True)
    assert b["best"] == a["best"] and b["measured"] < a["measured"]


@pytest.mark.parametrize("line", [False, True])
@pytest.mark.parametrize("seed", range(10))
def test_multimodal_local_optimum(seed, line):
    rng = np.random.default_rng(100 + seed)
    lat = sp.Lattice([list(range(5)), list(range(4)), list(range(3))],
                     predicate=lambda p: (p[0] + 2 * p[1] + p[2]) % 7 != 3)
    table = {p: float(rng.uniform()) for p in itertools.product(range(5), range(4), range(3))}
    calls = []

    def cost(idx):
        calls.append(lat.key(idx))
        return table[tuple(idx)]

    res = dr.droplet(lat, cost, budget=1000, line=line)
    best = res["best"]
    assert all(table[nb] >= table[best] for nb in lat.neighbors(best))
    assert table[best] >= min(table[p] for p in lat.valid_points())
    assert len(calls) == len(set(calls)) == res["measured"]
    meds = [table[p] for p in res["path"]]
    assert all(a > b for a, b in zip(meds, meds[1:]))
    assert all(lat.valid(p) for p in res["path"])


def test_frozen_axes():
    lat = sp.Lattice([list(range(4)), [0, 1]])
    cost = lambda p: (p[0] - 3) ** 2 + (0 if p[1] == 1 else 5)
    res = dr.droplet(lat, cost, start=(0, 0), frozen=(1,))
    assert res["best"] == (3, 0)
    assert dr.droplet(lat, cost, start=(0, 0))["best"] == (3, 1)


def test_failed_measurements_are_inf_and_counted():
    lat = sp.Lattice([list(range(5))])
    cost = lambda p: math.inf if p[0] == 1 else float(10 - p[0])
    res = dr.droplet(lat, cost, start=(0,))
    assert res["best"] == (0,) and res["measured"] == 2


@pytest.mark.parametrize("seed", range(20))
def test_ranksum_matches_scipy(seed):
    rng = np.random.default_rng(seed)
    n1, n2 = int(rng.integers(1, 15)), int(rng.integers(1, 15))
    a = np.round(rng.normal(1.0, 0.1, n1), 2)
    b = np.round(rng.normal(1.05, 0.1, n2), 2)
    if np.ptp(np.concatenate([a, b])) == 0:
        return
    ref = stats.mannwhitneyu(a, b, alternative="less", use_continuity=True,
                             method="asymptotic").pvalue
    assert dr.ranksum_p_less(list(a), list(b)) == pytest.approx(ref, rel=1e-12, abs=1e-15)


def test_statistical_convergence():
    lat = sp.Lattice([list(range(3))])
    noisy = {0: [1.00, 1.02, 0.98, 1.01, 0.99], 1: [0.99, 1.03, 0.97, 0.995, 1.01],
             2: [0.5, 0.52, 0.49, 0.51, 0.5]}
    res = dr.droplet(lat, lambda p: noisy[p[0]], start=(0,), alpha=0.05)
    assert res["best"] == (0,)            # median lower but not significant: stop
    res = dr.droplet(lat, lambda p: noisy[p[0]], start=(1,), alpha=0.05)
    assert res["best"] == (2,)
    res = dr.droplet(lat, lambda p: noisy[p[0]], start=(0,), alpha=1.0)
    assert [p[0] for p in res["path"]] == [0, 1, 2]      # deterministic: any lower median moves


def test_combined_explore_then_exploit():
    s = sp.Space(sp.OP_MATMUL, (1024, 1024, 1024))
    rng = np.random.default_rng(5)
    w = rng.uniform(0.5, 1.5, len(s.sizes))
    c = [rng.uniform(0, n - 1) for n in s.sizes]
    cost = lambda p: float(sum(wi * (i - ci) ** 2 for i, ci, wi in zip(p, c, w)))
    res = dr.combined(s, cost, seed=3, n_explore=300, budget=100)
    assert res["n_explore"] == 300 and res["n_droplet"] <= 100
    assert cost(res["best"]) <= min(cost(p) for p in res["samples"])
    assert cost(res["best"]) <= cost(res["seed_point"])
    best = res["best"]
    if res["status"] == dr.OK:
        assert all(cost(nb) >= cost(best) for nb in s.neighbors(best))
