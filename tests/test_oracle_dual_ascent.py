"""Pins of the oracle of the paper's approximate neuron assignment (Section 3, "Optimiser":
dual ascent on device offsets, a capacity fix-up, pairwise swaps).

What fixes it without an implementation to compare against:

* every result is balanced, and never beats the optimum found by brute force (small I) or
  by the exact solver;
* with two devices a balanced assignment that no swap improves is optimal, so the value
  equals the textbook two-device optimum (sort by M_k0 - M_k1, top half on device 0),
  written out here;
* at the end no single exchange of two neurons improves;
* when every neuron prefers one device and the preferences are already balanced, the
  offsets never move and the preferred assignment comes back unchanged;
* the fix-up moves exactly the excess neurons, each the cheapest one to move.
"""
import itertools

import numpy as np
import pytest

from oracle import dual_ascent as da
from oracle import layout as lay


def _random_M(I, L, seed, scale=1 << 40):
    rng = np.random.default_rng(seed)
    return rng.integers(0, scale, size=(I, L), dtype=np.int64)


def _brute_force(M):
    I, L = M.shape
    best = None
    for nu in itertools.product(range(L), repeat=I):
        if np.all(np.bincount(nu, minlength=L) == I // L):
            v = int(M[np.arange(I), list(nu)].sum())
            best = v if best is None else max(best, v)
    return best


@pytest.mark.parametrize("I,L,seed", [(12, 2, 0), (12, 3, 1), (8, 4, 2), (60, 3, 3), (256, 4, 4)])
def test_balanced_and_not_above_the_optimum(I, L, seed):
    M = _random_M(I, L, seed)
    nu, v = da.assign(M)
    assert np.all(np.bincount(nu, minlength=L) == I // L)
    assert v == int(M[np.arange(I), nu].sum())
    opt = _brute_force(M) if I <= 12 else lay.balanced_assign(M)[1]
    assert v <= opt


@pytest.mark.parametrize("I,seed", [(10, 5), (64, 6), (3072, 7)])
def test_two_devices_reach_the_sorted_optimum(I, seed):
    M = _random_M(I, 2, seed)
    _, v = da.assign(M)
    d = M[:, 0] - M[:, 1]
    order = np.argsort(-d, kind="stable")
    top = order[: I // 2]
    best = int(M[top, 0].sum() + np.delete(M[:, 1], top).sum())
    assert v == best


@pytest.mark.parametrize("I,L,seed", [(24, 3, 8), (32, 4, 9)])
def test_no_single_exchange_improves(I, L, seed):
    M = _random_M(I, L, seed)
    nu, _ = da.assign(M)
    for k1 in range(I):
        for k2 in range(k1 + 1, I):
            a, b = nu[k1], nu[k2]
            if a != b:
                assert M[k1, b] + M[k2, a] <= M[k1, a] + M[k2, b]


@pytest.mark.parametrize("I,L,seed", [(24, 3, 11), (40, 4, 12)])
def test_swaps_from_the_contiguous_layout_end_at_a_local_optimum(I, L, seed):
    """The swap phase alone, from the contiguous assignment: balanced, no better exchange."""
    M = _random_M(I, L, seed)
    start = np.repeat(np.arange(L), I // L)
    nu = da.pairwise_swaps(M, start)
    assert np.all(np.bincount(nu, minlength=L) == I // L)
    assert int(M[np.arange(I), nu].sum()) > int(M[np.arange(I), start].sum())
    for k1 in range(I):
        for k2 in range(k1 + 1, I):
            a, b = nu[k1], nu[k2]
            if a != b:
                assert M[k1, b] + M[k2, a] <= M[k1, a] + M[k2, b]


def test_balanced_preferences_come_back_unchanged():
    I, L = 12, 3
    pref = np.array([k % L for k in range(I)])
    M = np.zeros((I, L), dtype=np.int64)
    M[np.arange(I), pref] = 1000 + np.arange(I)
    lam, nu0 = da.dual_offsets(M)
    assert np.all(lam == 0.0)
    nu, v = da.assign(M)
    np.testing.assert_array_equal(nu, pref)
    assert v == int((1000 + np.arange(I)).sum())


def test_fix_up_moves_the_cheapest_excess():
    M = np.array([[9, 1], [5, 4], [7, 0], [3, 3]], dtype=np.int64)   # I = 4, L = 2
    nu = da.fix_up(M, np.array([0, 0, 0, 1]))
    # device 0 holds three neurons; the cheapest to move is neuron 1 (loss 5 - 4 = 1)
    np.testing.assert_array_equal(nu, [0, 1, 0, 1])
    M3 = _random_M(30, 3, 10)
    start = np.zeros(30, dtype=np.int64)
    start[25:] = 2                     # loads 25, 0, 5: 15 neurons must move
    moved = np.flatnonzero(da.fix_up(M3, start) != start)
    assert len(moved) == 15
