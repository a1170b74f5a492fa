"""Pins of the oracle's slot layout (generation-phase eviction that leaves kept
rows in place, Section 3): a worked example, and the properties that fix the
layout uniquely on random keep sets: it is a permutation of the keep set,
every kept row below C keeps its slot, and the kept rows at or past C fill the
other slots order-preservingly (the only increasing bijection between two
ascending lists).  A plausible mistake (movers in descending order, a mover
placed on a kept slot, a staying row moved, an off-by-one at C) fails one of
these."""

import numpy as np
import pytest

from oracle import slot_layout


def test_worked_example():
    # C = 5 slots, rows 0..6: rows 0, 2, 3 stay; rows 5 and 6 fill slots 1 and 4.
    assert slot_layout([0, 2, 3, 5, 6], 5).tolist() == [0, 5, 2, 3, 6]
    # Nothing past C kept: the identity.
    assert slot_layout([0, 1, 2, 3], 4).tolist() == [0, 1, 2, 3]
    # Every kept row past C: they fill slots 0..C-1 in order.
    assert slot_layout([7, 8, 11], 3).tolist() == [7, 8, 11]
    # Row C itself is a mover (the boundary), row C - 1 stays.
    assert slot_layout([1, 3, 4], 3).tolist() == [3, 1, 4]


def test_properties_on_random_sets():
    rng = np.random.default_rng(5)
    for _ in range(300):
        C = int(rng.integers(1, 40))
        m = int(rng.integers(0, 40))
        keep = np.sort(rng.choice(C + m, size=C, replace=False))
        out = slot_layout(keep, C)
        assert sorted(out.tolist()) == keep.tolist()                # a permutation of the keep set
        for r in keep[keep < C]:
            assert out[r] == r                                      # staying rows keep their slot
        free = [c for c in range(C) if c not in set(keep[keep < C].tolist())]
        movers = out[free]
        assert (movers >= C).all()                                  # free slots take rows past C
        assert (np.diff(movers) > 0).all()                          # in ascending order
        assert movers.tolist() == keep[keep >= C].tolist()


def test_rejects_a_list_that_is_not_an_ascending_set():
    with pytest.raises(AssertionError):
        slot_layout([2, 1, 3], 3)
    with pytest.raises(AssertionError):
        slot_layout([1, 1, 3], 3)
