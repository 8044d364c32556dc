"""The GPU-vs-oracle checkers themselves, on the CPU: each must reject the
mistakes it exists to catch (a selection cut short, an empty or duplicated
selection, a wrong assignment, a k-means run that leaves the oracle away from
a near-tie) and accept the near-tie cases the bands allow."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle  # noqa: E402
from parity_utils import check_assignment, check_kmeans_trajectory, selection_matches  # noqa: E402


def _case(seed=0, n=40):
    rng = np.random.default_rng(seed)
    a = rng.random(n)
    a /= a.sum()
    size = rng.integers(1, 30, n)
    return a, size


def test_selection_identical_is_not_excused():
    a, size = _case()
    ref, _ = oracle.select_budget(a, size, 200)
    assert selection_matches(a, size, 200, ref) is False


@pytest.mark.parametrize("cut", [1, 3])
def test_selection_truncated_fails(cut):
    a, size = _case()
    ref, _ = oracle.select_budget(a, size, 200)
    assert len(ref) > cut
    with pytest.raises(AssertionError, match="stops early"):
        selection_matches(a, size, 200, ref[:-cut])


def test_selection_empty_fails():
    a, size = _case()
    with pytest.raises(AssertionError):
        selection_matches(a, size, 200, [])


def test_selection_duplicate_and_range_fail():
    a, size = _case()
    ref, _ = oracle.select_budget(a, size, 200)
    with pytest.raises(AssertionError, match="twice"):
        selection_matches(a, size, 10 ** 6, ref + [ref[0]])
    with pytest.raises(AssertionError, match="range"):
        selection_matches(a, size, 10 ** 6, ref + [len(a)])


def test_selection_over_budget_and_wrong_unit_fail():
    a, size = _case()
    ref, tot = oracle.select_budget(a, size, 200)
    order = sorted(range(len(a)), key=lambda u: (-a[u], u))
    nxt = order[len(ref)]
    with pytest.raises(AssertionError):
        selection_matches(a, size, 200, ref + [nxt])
    # the lowest-scoring unit in place of a top one
    with pytest.raises(AssertionError):
        selection_matches(a, size, 200, ref[:-1] + [order[-1]])
    # rank order broken
    if len(ref) > 2:
        with pytest.raises(AssertionError, match="rank order"):
            selection_matches(a, size, 200, [ref[-1]] + ref[:-1])


def test_selection_near_tie_is_excused():
    a = np.array([0.3, 0.2, 0.2 * (1 + 1e-9), 0.1, 0.2 * (1 - 1e-7)])
    a = a / a.sum()
    size = np.array([5, 5, 5, 5, 9])
    ref, _ = oracle.select_budget(a, size, 15)
    assert ref == [0, 2, 1]
    assert selection_matches(a, size, 15, [0, 1, 2]) is True
    # a near-tied unit of another size taken in place of unit 1 leaves 1 token,
    # and the next unit (1, tied) does not fit: still a valid prefix stop
    assert selection_matches(a, size, 15, [0, 4]) is True
    # [0, 1] is valid too: a ranking with the tied unit 4 third stops there
    assert selection_matches(a, size, 15, [0, 1]) is True
    # without that tie, unit 1 alone after unit 0 leaves room for unit 2
    b = a.copy()
    b[4] = 0.01
    with pytest.raises(AssertionError, match="stops early"):
        selection_matches(b, size, 15, [0, 1])


def test_check_assignment_rejects_a_wrong_key_and_counts_ties():
    rng = np.random.default_rng(3)
    k = rng.standard_normal((200, 16))
    c = rng.standard_normal((8, 16))
    z = oracle.kmeans_assign(k, c)
    assert check_assignment(k, c, z) == 0
    bad = z.copy()
    d = ((k[0] - c) ** 2).sum(1)
    bad[0] = int(np.argsort(d)[-1])
    with pytest.raises(AssertionError):
        check_assignment(k, c, bad)
    c2 = c.copy()
    c2[5] = c2[2]
    z2 = oracle.kmeans_assign(k, c2)
    flip = z2.copy()
    flip[z2 == 2] = 5            # exact ties: either index is an argmin
    assert check_assignment(k, c2, flip) == int((z2 == 2).sum())


def _gpu_like(keys, init, n_iters, bf16, plant=None):
    """The oracle's own trajectory, as a GPU state callable, with an optional
    planted change at one iteration."""
    def state(it):
        res = oracle.kmeans(keys, init, it, bf16)
        z, c = res.z.copy(), res.centroids.copy()
        if plant is not None and it == plant[0]:
            plant[1](keys, z, c)
        return z, c
    return state


def test_kmeans_trajectory_accepts_the_oracle_and_rejects_plants():
    rng = np.random.default_rng(4)
    centres = rng.standard_normal((6, 16)) * 3
    keys = centres[rng.integers(0, 6, 300)] + rng.standard_normal((300, 16))
    init = rng.permutation(300)[:6]
    assert check_kmeans_trajectory(keys, init, 5, False, _gpu_like(keys, init, 5, False)) == 0
    assert check_kmeans_trajectory(keys, init, 5, True, _gpu_like(keys, init, 5, True)) == 0

    def wrong_key(k, z, c):
        z[7] = (z[7] + 1) % 6

    def shifted_centroid(k, z, c):
        c[2] += 1e-3

    for plant in (wrong_key, shifted_centroid):
        with pytest.raises(AssertionError):
            check_kmeans_trajectory(keys, init, 5, False, _gpu_like(keys, init, 5, False, (3, plant)))
