"""Pins of the reference whole-network trial split (Section 2.1, Termination in
Ansor; Section 3 setup: initial quota min(K/L, 64), the rest to the longest tasks)."""
import numpy as np
import pytest

from oracle import sampler as sa
from oracle import space as sp
from oracle import task_scheduler as ts


def lattice(n0=6, n1=5, n2=4):
    return sp.Lattice([list(range(n0)), list(range(n1)), list(range(n2))],
                      predicate=lambda p: (p[0] * 3 + p[1] + p[2]) % 5 != 2)


def const_cost(c):
    return lambda p: c + 1e-3 * (p[0] + p[1] + p[2])


@pytest.mark.parametrize("K,L,q", [(300, 24, 12), (10000, 24, 64), (1, 24, 1), (100, 13, 7),
                                   (25, 13, 1), (64 * 5, 5, 64)])
def test_initial_quota(K, L, q):
    lats = [lattice() for _ in range(L)]
    res = ts.tune_tasks(lats, [const_cost(1.0)] * L, [1] * L, list(range(L)), K, droplet_budget=0)
    assert res["quota"] == q
    assert res["rounds"][:L] == [(t, q) for t in range(L)]
    n_valid = len(lats[0].valid_points())
    assert res["spent"] == min(max(K, q * L), L * n_valid)    # every stream ends at n_valid


def test_streams_are_prefixes_of_the_sampler():
    lats = [lattice(), lattice(8, 3, 4), lattice(5, 5, 5)]
    seeds = [11, 22, 33]
    logs = [[], [], []]

    def mk(t, c):
        def cost(p):
            logs[t].append(tuple(p))
            return c + 1e-3 * sum(p)
        return cost

    res = ts.tune_tasks(lats, [mk(0, 3.0), mk(1, 1.0), mk(2, 2.0)], [1, 1, 1], seeds, 70,
                        droplet_budget=0)
    for t in range(3):
        n = res["tasks"][t]["n_explore"]
        assert logs[t] == sa.sample(lats[t], seeds[t], n)


def test_remaining_trials_go_to_the_longest_weighted_task():
    lats = [lattice(), lattice(), lattice()]
    # task 0 runs 10 units, task 1 runs 1, task 2 runs 4: the extra rounds all go
    # to task 0 while its stream lasts.
    res = ts.tune_tasks(lats, [const_cost(10.0), const_cost(1.0), const_cost(4.0)], [1, 1, 1],
                        [1, 2, 3], 60, droplet_budget=0)
    assert res["quota"] == 20
    assert res["rounds"] == [(0, 20), (1, 20), (2, 20)]
    res = ts.tune_tasks(lats, [const_cost(10.0), const_cost(1.0), const_cost(4.0)], [1, 1, 1],
                        [1, 2, 3], 100, droplet_budget=0)
    assert res["quota"] == 33
    assert res["rounds"] == [(0, 33), (1, 33), (2, 33), (0, 1)]
    # weights: task 1 occurs 20 times, so it is the longest (20 > 10 > 4)
    res = ts.tune_tasks(lats, [const_cost(10.0), const_cost(1.0), const_cost(4.0)], [1, 20, 1],
                        [1, 2, 3], 40, droplet_budget=0)
    assert res["rounds"] == [(0, 13), (1, 13), (2, 13), (1, 1)]


def test_exhausted_task_leaves_the_worklist():
    tiny = sp.Lattice([[0, 1, 2]])
    big = lattice()
    res = ts.tune_tasks([tiny, big], [lambda p: 100.0 + p[0], const_cost(1.0)], [1, 1], [5, 6],
                        40, droplet_budget=0)
    assert res["tasks"][0]["n_explore"] == 3
    assert res["spent"] == 40 and res["tasks"][1]["n_explore"] == 37
    assert res["rounds"][:2] == [(0, 3), (1, 20)]


def test_network_time_and_droplet_per_task():
    lats = [lattice(), lattice(7, 6, 5)]
    rng = np.random.default_rng(0)
    centers = [rng.uniform(0, 4, 3), rng.uniform(0, 4, 3)]
    costs = [lambda p, c=c: 1.0 + float(sum((i - ci) ** 2 for i, ci in zip(p, c))) for c in centers]
    res = ts.tune_tasks(lats, costs, [3, 2], [7, 8], 20, droplet_budget=100)
    net = 0.0
    for t in range(2):
        tk = res["tasks"][t]
        assert tk["best_time"] <= tk["explore_time"]
        assert tk["n_droplet"] <= 101
        net += [3, 2][t] * tk["best_time"]
    assert res["network_time"] == pytest.approx(net, rel=0, abs=0)
