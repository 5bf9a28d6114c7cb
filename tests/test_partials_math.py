"""Bookkeeping of the per-workgroup histograms, by brute force (no GPU).

The scoring pass splits T = units x groups-per-unit groups of keys into nwg
contiguous ranges, [wg*T/nwg, (wg+1)*T/nwg).  A workgroup stores the
histogram of each unit it meets as slot unit + wg (zeros when its groups of
the unit all lie past n_b), and the selection of a unit sums the slots of the
workgroups that own its first and last group and every one between.  These
checks enumerate the ranges directly; the selection's reading is the case
where every group of the unit counts.
Slots must be unique.  The owner of a group, computed as
((g + 1) * nwg - 1) // T, must be the range that holds it.  The workgroups
between the two owners must be exactly those whose range meets the unit's
valid groups.  And the bound the library uses to pick this mode,
ceil(gu / floor(T / nwg)) + 1, must cover the slot count of every unit.
"""
from __future__ import annotations

import numpy as np
import pytest


def owner(g, T, nwg):
    return ((g + 1) * nwg - 1) // T


def ranges(T, nwg):
    return [(T * wg // nwg, T * (wg + 1) // nwg) for wg in range(nwg)]


CASES = [(1, 1, 1), (2, 5, 3), (128, 1024, 512), (128, 94, 512), (256, 47, 512), (16, 7, 100),
         (3, 1000, 7), (64, 4096, 1024), (5, 3, 15)]


@pytest.mark.parametrize("U,gu,nwg", CASES)
def test_owner_and_slots(U, gu, nwg):
    T = U * gu
    nwg = min(nwg, T)  # the grid never has more workgroups than groups
    rs = ranges(T, nwg)
    assert rs[0][0] == 0 and rs[-1][1] == T
    assert all(a < b for a, b in rs), "every range holds a group"
    for wg, (a, b) in enumerate(rs):
        for g in range(a, b):
            assert owner(g, T, nwg) == wg
    slots = set()
    for wg, (a, b) in enumerate(rs):
        for u in range(a // gu, (b - 1) // gu + 1):  # units this range meets
            s = u + wg
            assert s not in slots, (u, wg)
            slots.add(s)
    assert max(slots) < U + nwg


@pytest.mark.parametrize("U,gu,nwg", CASES)
def test_select_covers_the_writers(U, gu, nwg):
    T = U * gu
    nwg = min(nwg, T)
    rs = ranges(T, nwg)
    shortest = T // nwg
    bound = -(-gu // shortest) + 1
    rng = np.random.default_rng(U * 7 + gu)
    for u in range(U):
        g0 = u * gu
        for vg in sorted({1, gu, int(rng.integers(1, gu + 1))}):  # valid groups of the unit
            lo, hi = owner(g0, T, nwg), owner(g0 + vg - 1, T, nwg)
            writers = [wg for wg, (a, b) in enumerate(rs) if a < g0 + vg and b > g0]
            assert writers == list(range(lo, hi + 1)), (u, vg)
            assert hi - lo + 1 <= bound, (u, vg, hi - lo + 1, bound)
