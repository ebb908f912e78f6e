"""Reference whole-network budget split across layers (test infrastructure only).

Section 2.1 ("Termination in Ansor") and Section 3 (experimental setup): a
network of L kernels (tasks) is tuned with one budget of K trials.  Every task
first receives ``min(K/L, 64)`` trials in round-robin order; the remaining
trials go to the tasks that account for the longest running time.  The best
schedule of each task is then handed to Droplet Search, which runs per task to
convergence (or its own budget).

Readings where the paper is loose:

* The initial quota is ``q = max(1, min(K // L, 64))`` -- at least one trial
  per task, so a budget below L still yields a schedule for every task (the
  total then exceeds K).
* A task's trials are the next points of its own exploration stream (the
  sampler of ``oracle.sampler`` with that task's seed), so that a task given
  ``n`` trials over several rounds measures exactly the first ``n`` points of
  ``sample(space, seed, n)``.
* After the initial round, while fewer than K trials were spent, the task with
  the largest weighted time ``weight * best_time`` (ties: lowest index) whose
  stream is not exhausted receives ``min(q, K - spent)`` more trials; a task
  whose stream ends is dropped from the worklist.  The weight is the number of
  times the kernel occurs in the network.
* The network time is ``sum(weight * best_time)`` over the tasks.

Pins (tests/test_oracle_task_scheduler.py): quotas and totals worked by hand,
the prefix property of the streams, and the longest-task rule on costs chosen
so the order of allocations is known in advance.
"""
from __future__ import annotations

import math

from .droplet import Meas, droplet
from .sampler import Stream


class _Stream:
    """The exploration sampler's draw sequence, consumed incrementally."""

    def __init__(self, space, seed):
        self.stream = Stream(space, seed)
        self.taken = 0
        self.ended = False

    def take(self, n):
        out = []
        while len(out) < n:
            p = self.stream.next()
            if p is None:
                self.ended = True
                break
            out.append(p)
        self.taken += len(out)
        return out


def tune_tasks(spaces, costs, weights, seeds, total_trials, droplet_budget=100, alpha=1.0):
    """Returns dict(tasks=[...], rounds=[(task, n)], spent, network_time)."""
    L = len(spaces)
    q = max(1, min(total_trials // L, 64)) if L else 0
    streams = [_Stream(sp, sd) for sp, sd in zip(spaces, seeds)]
    caches = [dict() for _ in range(L)]
    best = [None] * L
    best_t = [math.inf] * L
    n_trials = [0] * L
    rounds = []
    spent = 0

    def run_round(t, n):
        nonlocal spent
        pts = streams[t].take(n)
        for p in pts:
            m = Meas.of(costs[t](p))
            caches[t][spaces[t].key(p)] = m
            if best[t] is None or m.median < best_t[t]:
                best[t], best_t[t] = p, m.median
        n_trials[t] += len(pts)
        spent += len(pts)
        rounds.append((t, len(pts)))

    for t in range(L):
        run_round(t, q)
    while spent < total_trials:
        live = [t for t in range(L) if not streams[t].ended and best[t] is not None]
        if not live:
            break
        pick = live[0]
        for t in live[1:]:
            if weights[t] * best_t[t] > weights[pick] * best_t[pick]:
                pick = t
        run_round(pick, min(q, total_trials - spent))
    tasks = []
    for t in range(L):
        if best[t] is None:
            tasks.append(dict(best=None, explore_best=None, n_explore=0, n_droplet=0))
            continue
        d = droplet(spaces[t], costs[t], start=best[t], budget=droplet_budget, alpha=alpha,
                    cache=caches[t])
        tasks.append(dict(best=d["best"], best_time=d["meas"].median, explore_best=best[t],
                          explore_time=best_t[t], n_explore=n_trials[t], n_droplet=d["measured"]))
    net = sum(w * tk["best_time"] for w, tk in zip(weights, tasks) if tk["best"] is not None)
    return dict(tasks=tasks, rounds=rounds, spent=spent, quota=q, network_time=net)
