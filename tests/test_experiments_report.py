"""The experiment report (no GPU): markdown tables built from the JSON lines
that the exploitation comparison (Section 3, RQ4), the exploration sweep (RQ5)
and the network trial split (Section 2.1) print."""
import json

from paper_2406_20037_amd import experiments as E


def _write(tmp_path, rows):
    p = tmp_path / "rows.jsonl"
    p.write_text("".join(json.dumps(r) + "\n" for r in rows))
    return str(p)


def test_report_tables(tmp_path):
    ex = [dict(experiment="exploiters", workload="w", seed=s, n_explore=300, seed_us=10.0 + s,
               strategy=st, valid_only=vo, best_us=b, measured=m, failed=f, exploit_s=0.5)
          for s, st, vo, b, m, f in [(1, "droplet", 0, 9.0, 12, 0), (2, "droplet", 0, 8.0, 20, 0),
                                     (1, "ga", 1, 9.5, 100, 0), (2, "ga", 1, 8.5, 100, 0)]]
    sw = [dict(experiment="sweep", workload="w", seed=1, n_explore=n, n_explore_measured=n,
               n_droplet_measured=d, best_us=b, explore_s=0.1, droplet_s=0.2)
          for n, d, b in [(10, 30, 9.0), (1, 50, 12.0)]]
    sw.append(dict(experiment="sweep", workload="w", seed=9, n_explore=10000,
                   n_explore_measured=6236, n_droplet_measured=0, random_only=True, best_us=7.0,
                   explore_s=3.0))
    ts = [dict(experiment="tasks", workload="net", total_trials=24, quota=1, rounds=24,
               droplet_trials=100, network_us=1234.56, wall_s=2.0, per_task=[{}] * 24)]
    text = E.report([_write(tmp_path, ex + sw + ts)])
    lines = text.splitlines()
    assert "w: 2 seeds, best of 300 samples 11.50 us (mean)" in lines
    assert "| droplet | count | 8.50 | 9.00 / 8.00 | 12 / 20 | 0 / 0 | 0.50 |" in lines
    assert "| ga | skipped | 9.00 | 9.50 / 8.50 | 100 / 100 | 0 / 0 | 0.50 |" in lines
    # sweep rows come out in increasing N, the random-only row last
    i1, i10 = lines.index("| 1 | 12.00 | 12.00 | 50 | 0.10 | 0.20 |"), \
        lines.index("| 10 | 9.00 | 9.00 | 30 | 0.10 | 0.20 |")
    i10k = lines.index("| 10000 (random only, 6236 points) | 7.00 | 7.00 | 0 | 3.00 | 0.00 |")
    assert i1 < i10 < i10k
    assert "| 24 | 1 | 24 | 100 | 1234.6 | 2.0 |" in lines
