"""Pins of the reference sampler and of the shared input generator."""
import numpy as np
import pytest
from scipy import stats

import synthdata
from oracle import sampler as sm
from oracle import space as sp

# Published SplitMix64 outputs for seed 1234567 (the reference sequence of the
# generator's definition, also used by the Rosetta Code task on SplitMix64).
SEQ_1234567 = [6457827717110365317, 3203168211198807973, 9817491932198370423,
               4593380528125082431, 16408922859458223821]


def test_splitmix64_published_sequence():
    g = sm.SplitMix64(1234567)
    assert [g.next() for _ in range(5)] == SEQ_1234567
    assert [int(v) for v in synthdata.splitmix64(1234567, 5)] == SEQ_1234567
    assert [int(v) for v in synthdata.splitmix64(1234567, 2, start=3)] == SEQ_1234567[3:]


def test_uniform_and_ints_ranges():
    u = synthdata.uniform(1, (100000,))
    assert u.dtype == np.float32 and u.min() >= -1.0 and u.max() < 1.0
    assert abs(float(u.mean())) < 0.01
    # every value is k / 2**23 - 1 exactly
    assert np.array_equal((u.astype(np.float64) + 1.0) * 2 ** 23, np.round((u + 1.0) * 2 ** 23))
    i = synthdata.small_int(2, (100000,), 8)
    assert set(np.unique(i).tolist()) == set(range(-8, 9))
    n = synthdata.normal(3, (200000,))
    assert abs(float(n.mean())) < 0.01 and abs(float(n.std()) - 1.0) < 0.01


def test_below_uniform_chi_square():
    for n in (3, 5, 6, 7):
        g = sm.SplitMix64(99 + n)
        counts = np.bincount([g.below(n) for _ in range(20000)], minlength=n)
        assert stats.chisquare(counts).pvalue > 0.01


def test_sample_determinism_distinct_valid():
    s = sp.Space(sp.OP_CONV, (1, 64, 56, 56, 64, 3, 3, 1, 1))
    a = sm.sample(s, 7, 300)
    assert a == sm.sample(s, 7, 300) and a != sm.sample(s, 8, 300)
    assert len(a) == 300 and len(set(a)) == 300 and all(s.valid(p) for p in a)


def test_sample_exhausts_small_lattice():
    lat = sp.Lattice([[0, 1, 2, 3], [0, 1, 2, 3], [0, 1, 2]], predicate=lambda p: sum(p) % 5 != 0)
    got = sm.sample(lat, 1, 300)
    assert sorted(got) == sorted(lat.valid_points())
    empty = sp.Lattice([[0, 1]], predicate=lambda p: False)
    assert sm.sample(empty, 1, 10) == []


def test_first_draw_uniform_over_lattice():
    lat = sp.Lattice([[0, 1, 2], [0, 1, 2, 3, 4]])
    firsts = [lat.key(sm.sample(lat, seed, 1)[0]) for seed in range(6000)]
    counts = np.bincount(firsts, minlength=15)
    assert stats.chisquare(counts).pvalue > 0.01


class _FamilySpace(sp.Lattice):
    """A small space with a kernel-family axis: family 0 has 12 valid
    points, family 1 has 3, family 2 none."""
    op = 0

    def __init__(self):
        super().__init__([[0, 1, 2], [0, 1, 2, 3], [0, 1, 2]], names=["a", "b", "mfma"],
                         predicate=lambda p: p[2] == 0 or (p[2] == 1 and p[1] == 0))


def test_first_draw_uniform_over_families_then_within():
    s = _FamilySpace()
    firsts = [sm.sample(s, seed, 1)[0] for seed in range(6000)]
    fam = np.bincount([p[2] for p in firsts], minlength=3)
    assert fam[2] == 0 and stats.chisquare(fam[:2]).pvalue > 0.01
    for f, n in ((0, 12), (1, 3)):
        within = [s.key(p) for p in firsts if p[2] == f]
        counts = np.unique(within, return_counts=True)[1]
        assert len(counts) == n and stats.chisquare(counts).pvalue > 0.01


def test_families_drawn_until_exhausted():
    s = _FamilySpace()
    got = sm.sample(s, 5, 100)
    assert sorted(got) == sorted(s.valid_points()) and len(got) == 15
    # the small family is used up after a few draws; the rest come from family 0
    assert sum(1 for p in got[:6] if p[2] == 1) >= 1

