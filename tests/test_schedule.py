"""Pins of the oracle's block schedule against published definitions and invariants."""

import itertools
import os

import numpy as np
import pytest

from oracle import schedule

HERE = os.path.dirname(os.path.abspath(__file__))


def test_splitmix64_published_outputs():
    """First outputs of SplitMix64 from state 0, as published with the reference code."""
    with open(os.path.join(HERE, "golden", "splitmix64_seed0.txt")) as f:
        want = [int(line, 16) for line in f if line.strip() and not line.startswith("#")]
    g = schedule.SplitMix64(0)
    assert [g.next() for _ in range(len(want))] == want


def test_lemire_power_of_two_takes_top_bits():
    """For k = 2^b the multiply-shift method never rejects and returns the top b bits."""
    for b in (1, 3, 10, 31, 63):
        g1, g2 = schedule.SplitMix64(77), schedule.SplitMix64(77)
        for _ in range(200):
            assert schedule.bounded(g1, 1 << b) == g2.next() >> (64 - b)


def test_lemire_range_and_uniformity():
    g = schedule.SplitMix64(123)
    for k in (1, 2, 3, 5, 17, 1000):
        vals = [schedule.bounded(g, k) for _ in range(3000)]
        assert min(vals) >= 0 and max(vals) < k
    counts = np.bincount([schedule.bounded(g, 3) for _ in range(30000)], minlength=3)
    chi2 = np.sum((counts - 10000) ** 2 / 10000)
    assert chi2 < 13.8  # p = 0.001 at 2 degrees of freedom


def test_shuffle_is_uniform_permutation():
    perms = list(itertools.permutations(range(3)))
    counts = dict.fromkeys(perms, 0)
    for s in range(6000):
        p = tuple(schedule.shuffled(schedule.SplitMix64(s * 7919 + 1), 3))
        counts[p] += 1
    chi2 = sum((c - 1000) ** 2 / 1000 for c in counts.values())
    assert chi2 < 20.5  # p = 0.001 at 5 degrees of freedom
    for k in (1, 2, 17, 64):
        p = schedule.shuffled(schedule.SplitMix64(k), k)
        assert sorted(p) == list(range(k))


@pytest.mark.parametrize("R,C", [(4, 4), (8, 8), (17, 17), (31, 7), (7, 31), (1, 1), (1, 5), (3, 1)])
def test_interleave_invariants(R, C):
    for t in range(5):
        s = schedule.sweep_schedule(99, t, R, C, True)
        w = [x - 1 for x in s if x > 0]
        h = [-x - 1 for x in s if x < 0]
        assert sorted(w) == list(range(C)) and sorted(h) == list(range(R))
        assert (s[0] > 0) == (C >= R)
        if R == C:
            assert all((x > 0) == (i % 2 == 0) for i, x in enumerate(s))
        # proportional: after any prefix the W share tracks C / (R + C) within one step
        nw = np.cumsum([x > 0 for x in s])
        k = np.arange(1, len(s) + 1)
        assert np.all(np.abs(nw - k * C / (R + C)) <= 1.0 + 1e-12)


def test_schedule_depends_on_seed_and_sweep_and_deterministic_listing():
    a = schedule.sweep_schedule(5, 0, 8, 8)
    assert a == schedule.sweep_schedule(5, 0, 8, 8)
    assert a != schedule.sweep_schedule(5, 1, 8, 8)
    assert a != schedule.sweep_schedule(6, 0, 8, 8)
    assert schedule.sweep_schedule(5, 3, 3, 2, False) == [1, 2, -1, -2, -3]
