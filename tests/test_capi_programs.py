"""The compiled program each valid schedule selects (host only, no GPU).

Two valid points of a workload's lattice launch the same program when they
select the same template instance with the same kernel-argument block.  The
only such pairs allowed are points that differ in the unroll knob alone and
whose unroll values give the same effective factor (the saturation of TVM's
auto_unroll_max_step reading: e.g. unroll 64 and 512 over one accumulator per
step both unroll 16 times); every other knob must change the program.  The
oracle's geometry gives the effective factor independently.
"""
import numpy as np
import pytest

from synthdata import workloads as wl
from oracle import space as osp
from paper_2406_20037_amd import _lib as lib

TASKS = ([(n, op, sh) for n, (op, sh) in wl.SINGLE.items()] +
         [(n, op, sh) for n, op, sh, _ in wl.RESNET50] +
         [("vgg_" + n, op, sh) for n, op, sh, _ in wl.VGG16])


@pytest.mark.parametrize("name,op,sh", TASKS, ids=[t[0] for t in TASKS])
def test_identical_programs_differ_only_in_a_saturated_unroll(name, op, sh):
    c = lib.Space(op, sh)
    keys, inst, hashes = c.programs()
    assert len(keys) > 0
    ua = c.names.index("unroll")
    radix = int(np.prod([len(v) for v in c.values[:ua]]))
    nu = len(c.values[ua])
    digit = (keys // np.uint64(radix)) % np.uint64(nu)
    rest = keys - digit * np.uint64(radix)           # the key with unroll at index 0
    prog = inst.astype(np.uint64) * np.uint64(1 << 20) ^ hashes
    order = np.lexsort((rest, prog))
    same = prog[order][1:] == prog[order][:-1]
    # within one program, every point has the same key apart from unroll
    assert np.array_equal(rest[order][1:][same], rest[order][:-1][same]), name
    # conversely, points with the same other knobs and different programs
    # differ in the effective unroll factor: check a sample against the oracle
    o = osp.Space(op, sh)
    rng = np.random.default_rng(len(keys))
    pick = rng.choice(len(order) - 1, size=min(300, len(order) - 1), replace=False)
    for i in pick:
        a, b = int(keys[order[i]]), int(keys[order[i + 1]])
        ga, gb = o.geometry(o.from_key(a)), o.geometry(o.from_key(b))
        if same[i]:
            assert ga["unroll_eff"] == gb["unroll_eff"] and ga["t0"] == gb["t0"]
    # for a sample of the other knobs' settings, the library's distinct
    # programs over the unroll values are as many as the oracle's distinct
    # effective factors
    uniq_rest = np.unique(rest)
    for r in rng.choice(uniq_rest, size=min(200, len(uniq_rest)), replace=False):
        pts = [int(r) + d * radix for d in range(nu)]
        valid = [k for k in pts if o.valid(o.from_key(k))]
        eff = {o.geometry(o.from_key(k))["unroll_eff"] for k in valid}
        progs = {int(prog[np.searchsorted(keys, np.uint64(k))]) for k in valid}
        assert len(progs) == len(eff), (name, o.knobs(o.from_key(int(r))))
