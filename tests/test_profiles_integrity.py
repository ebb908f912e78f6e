"""The committed profile summaries (no GPU): every profiled schedule is a valid
point of its workload's lattice (a point outside it would be refused by the
profiling driver, and a summary made of such a run holds no kernel of ours),
every summary's kernel trace lists at least one kernel of the library's
families, and every HBM-traffic entry was made by a command one of the
summaries gives."""
import json
import pathlib
import re

from oracle import space as S
from synthdata import workloads as wl

ROOT = pathlib.Path(__file__).resolve().parent.parent
PROFILES = ROOT / "profiles"
CMD = re.compile(r"prof_run --workload (\S+) --sched (\S+)")
OURS = re.compile(r"^\| `(conv_valu|conv_mfma2?|mm_valu|mm_mfma|split_reduce_kernel|"
                  r"mfma_ceiling_kernel)[<(]")


def resolve(workload):
    if workload.startswith("conv:"):
        return wl.OP_CONV, tuple(int(v) for v in workload[5:].split(","))
    if ":" in workload:
        net, layer = workload.split(":", 1)
        table = {"resnet50": wl.RESNET50, "vgg16": wl.VGG16}[net]
        return next((op, sh) for name, op, sh, _ in table if name == layer)
    return wl.SINGLE[workload]


def summaries():
    files = sorted(PROFILES.glob("*.md"))
    assert files, "no profile summaries"
    return files


def test_every_profiled_schedule_is_valid():
    seen = 0
    for f in summaries():
        for workload, sched in set(CMD.findall(f.read_text())):
            op, shape = resolve(workload)
            sp = S.Space(op, shape)
            knobs = dict(kv.split("=") for kv in sched.split(","))
            assert sorted(knobs) == sorted(sp.names), (f.name, sched)
            idx = [sp.values[a].index(int(knobs[n])) for a, n in enumerate(sp.names)]
            assert sp.valid(idx), (f.name, workload, sched)
            seen += 1
    assert seen >= 20


def test_every_trace_lists_a_kernel_of_ours():
    for f in summaries():
        text = f.read_text()
        if "### Kernel trace" not in text:
            continue
        trace = text.split("### Kernel trace", 1)[1].split("###", 1)[0]
        rows = [l for l in trace.splitlines() if OURS.match(l)]
        assert rows, f.name


def test_traffic_entries_come_from_committed_commands():
    traffic = json.loads((PROFILES / "traffic.json").read_text())
    commands = set()
    for f in summaries():
        commands.update(CMD.findall(f.read_text()))
    assert traffic
    for key, entry in traffic.items():
        m = CMD.search(entry["command"])
        assert m, key
        assert m.groups() in commands, key
        assert entry["read_bytes"] > 0 and entry["write_bytes"] > 0, key
