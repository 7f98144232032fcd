"""Pins of the oracle's anchor selection (Sec. 3.1): hand-worked calibration sets,
the tie and fallback rules, and invariances of standardised scores."""
import random

import pytest

from oracle import anchors


def test_hand_worked_set_strict_median():
    # L mean 13.2, population sd 18.734; Theta mean 0.184, sd 0.14623; median Theta 0.3.
    # z-sums: clip 0 -1.963 (smallest), clip 1 -1.841.  Only clip 4 (0.31) lies strictly above
    # the median (with ">=" clips 2 and 3 would join and clip 2, product 1.558, would win).
    L = [0.0, 1.0, 50.0, 10.0, 5.0]
    Th = [0.0, 0.01, 0.3, 0.3, 0.31]
    assert anchors.select_anchors(L, Th, 1e-6) == (0, 4)


def test_hand_worked_set_largest_product():
    # L mean 21, sd 14.967; Theta mean 0.24, sd 0.18547; median 0.2.  Candidates above the
    # median: clip 2 (z 1.270, 1.402: product 1.780) and clip 3 (z -0.067, 0.863: -0.058).
    L = [0.0, 10.0, 40.0, 20.0, 35.0]
    Th = [0.0, 0.1, 0.5, 0.4, 0.2]
    assert anchors.select_anchors(L, Th, 1e-6) == (0, 2)


def test_median_of_even_count_and_population_sd():
    assert anchors.median([4.0, 1.0, 3.0, 2.0]) == 2.5
    assert anchors.median([5.0, 1.0, 3.0]) == 3.0
    # population sd of (0, 2) is 1: z = (-1, 1)
    assert anchors.standardise([0.0, 2.0], 1e-6) == [-1.0, 1.0]
    # zero spread: the denominator is eps
    assert anchors.standardise([3.0, 3.0, 3.0], 0.5) == [0.0, 0.0, 0.0]


def test_ties_keep_the_lower_index():
    L = [0.0, 0.0, 10.0, 10.0]
    Th = [0.0, 0.0, 1.0, 1.0]
    assert anchors.select_anchors(L, Th, 1e-6) == (0, 2)


def test_fallback_when_no_clip_qualifies():
    # every Theta equal: none lies above the median
    assert anchors.select_anchors([0.0, 5.0, 9.0], [0.2, 0.2, 0.2], 1e-6)[1] is None
    # the only turning clip travels less than the low-motion anchor
    i0, i1 = anchors.select_anchors([5.0, 0.0], [0.0, 1.0], 1e-6)
    assert i0 == 0 and i1 is None
    # a single clip is its own low-motion anchor and nothing is above it
    assert anchors.select_anchors([3.0], [0.1], 1e-6) == (0, None)


def test_stationary_and_moving_turn_pair():
    # a stationary clip, straight clips and one fast turn: the turn is the moving anchor
    L = [0.0, 20.0, 20.0, 18.0]
    Th = [0.0, 0.0, 0.01, 0.6]
    assert anchors.select_anchors(L, Th, 1e-6) == (0, 3)


def _random_set(rng, n):
    # well-separated values (no near-ties), so exact rescaling cannot flip a comparison
    L = [rng.randrange(0, 4000) * 0.01 + i * 1e-4 for i in range(n)]
    Th = [rng.randrange(0, 600) * 0.001 + i * 1e-6 for i in range(n)]
    return L, Th


def test_invariant_to_power_of_two_scaling():
    rng = random.Random(11)
    for _ in range(200):
        L, Th = _random_set(rng, rng.randrange(2, 12))
        want = anchors.select_anchors(L, Th, 1e-12)
        for s in (0.25, 2.0, 8.0):
            assert anchors.select_anchors([s * v for v in L], [s * v for v in Th], 1e-12) == want


@pytest.mark.parametrize("n", [3, 6, 11])
def test_clip_order_does_not_matter_without_ties(n):
    rng = random.Random(n)
    for _ in range(100):
        L, Th = _random_set(rng, n)
        i0, i1 = anchors.select_anchors(L, Th, 1e-12)
        perm = list(range(n))
        rng.shuffle(perm)
        j0, j1 = anchors.select_anchors([L[p] for p in perm], [Th[p] for p in perm], 1e-12)
        assert perm[j0] == i0
        assert (j1 is None and i1 is None) or perm[j1] == i1
