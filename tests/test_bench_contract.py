"""bench.py's output contract: one JSON line with the headline metric, the
roofline of the dominant kernel and the oracle's CPU rate; more than one GPU is
refused before anything touches a device."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    assert "one GPU" in capsys.readouterr().err


@pytest.mark.gpu
def test_json_line_contract():
    cmd = [sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workloads", "vgg16",
           "--layers", "0-1", "--steps", "2", "--warmup", "1", "--n-explore", "30",
           "--budget", "10"]
    print("bench:", " ".join(cmd[2:]), flush=True)
    r = subprocess.run(cmd, cwd=ROOT, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True,
                       timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, r.stdout[-2000:]
    d = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
              "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
              "roofline", "cpu_baseline"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 2 and d["warmup"] == 1
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["higher_is_better"] is True
    assert d["unit"] == "GFLOP/s" and d["dtype"] == "f32" and d["vs_baseline"] is None
    # value is the pass's algorithmic flop over its mean time
    from synthdata import workloads as wl
    tasks = [c for c in d["configs"] if c["name"] == "vgg16"][0]["tasks"]
    assert [t["name"] for t in tasks] == d["config"]["layers"]
    flop = sum(t["count"] * wl.flops(wl.OP_CONV, t["shape"]) for t in tasks)
    assert d["value"] == pytest.approx(flop / (d["ms_per_step"] * 1e-3) / 1e9, rel=2e-3)
    assert "workload" in d["config"] and "VGG-16" in d["config"]["workload"]
    rl = d["roofline"]
    for k in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert k in rl, k
    assert rl["bound"] in ("mfma", "hbm", "alu")
    assert rl["frac"] == pytest.approx(rl["achieved"] / rl["peak"], rel=1e-3)
    assert 0 < rl["frac"] < 1
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["value"] > 0 and cpu["cores"] >= 1 and cpu["sample"]
    assert d["parity"]["status"] == "ok" and d["parity"]["max_rel_err"] <= 1e-4
