"""Pins of the oracle's slicing DP (Sec. 3.3, Eq. 5-8, Algorithm 1).

* Exhaustive enumeration of every slicing (2^(U-1) compositions) gives the
  same optimal latency, and the DP's slicing is one of the optimal ones.
* Closed forms: costs linear in the slice length with no context term give
  unit slices for K >= 2 and one slice for K = 1 with a fixed per-slice cost.
* The worked example after Eq. 5 (K = 4: T = t1 + ... + t4 + 3 t4).
* The eps rule: the answer is within K * eps of the optimum.
"""
import os

import numpy as np
import pytest

from oracle import dp_optimal_slicing, eq5_latency, exhaustive_optimal
from oracle.oracle import slicing_costs
from paper_2102_07988_amd import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("kind", ["random", "ties", "linear", "flops"])
@pytest.mark.parametrize("K", [1, 2, 3, 4, 8])
def test_dp_equals_exhaustive(kind, K):
    U = 12
    for seed in range(3):
        cost = synth.cost_table(U, kind, seed)
        best, argmins = exhaustive_optimal(cost, K)
        units, T, tmax, _ = dp_optimal_slicing(cost, K)
        assert sum(units) == U
        assert T == best, (kind, K, seed)
        assert tuple(units) in argmins
        assert eq5_latency(slicing_costs(cost, units), K) == T
        assert max(slicing_costs(cost, units)) <= tmax


def test_dp_small_sizes_exhaustive():
    for U in range(1, 10):
        for seed in range(4):
            cost = synth.cost_table(U, "random", 100 + seed)
            for K in (1, 2, 5):
                best, argmins = exhaustive_optimal(cost, K)
                units, T, _, _ = dp_optimal_slicing(cost, K)
                assert T == best and tuple(units) in argmins


def test_closed_form_linear_no_context():
    """t(n, c) = alpha * n: every slicing sums to alpha * L, so Eq. 5 is minimised by
    the smallest maximum, i.e. all slices one unit: T = alpha L + (K-1) alpha."""
    U, alpha = 16, 7
    cost = np.fromfunction(lambda k, j: alpha * (k + 1), (U, U), dtype=np.int64).astype(np.int64)
    for K in (2, 3, 48):
        units, T, _, _ = dp_optimal_slicing(cost, K)
        assert units == [1] * U
        assert T == alpha * U + (K - 1) * alpha


def test_closed_form_single_slice_for_one_cell():
    """K = 1 and t(n, c) = beta + alpha n with beta > 0: one slice is optimal, T = beta + alpha L."""
    U, alpha, beta = 16, 3, 50
    cost = np.fromfunction(lambda k, j: beta + alpha * (k + 1), (U, U), dtype=np.int64).astype(np.int64)
    units, T, _, _ = dp_optimal_slicing(cost, 1)
    assert units == [U]
    assert T == beta + alpha * U


def test_eq5_worked_example():
    rows = [list(map(int, ln.split())) for ln in open(os.path.join(GOLD, "eq5_example.txt"))
            if ln.strip() and not ln.startswith("#")]
    for K, t1, t2, t3, t4, T in rows:
        assert eq5_latency([t1, t2, t3, t4], K) == T


def test_eps_bound_and_identity():
    """With eps the answer is within K * eps of the optimum; eps = 0 is exact."""
    U = 12
    for seed in range(5):
        cost = synth.cost_table(U, "linear", seed)
        for K in (2, 4, 8):
            _, T0, _, ev0 = dp_optimal_slicing(cost, K, 0)
            for eps in (1, 5, 20, 100):
                _, Te, _, eve = dp_optimal_slicing(cost, K, eps)
                assert T0 <= Te <= T0 + K * eps
                assert eve <= ev0


def test_early_stop_evaluates_fewer_thresholds():
    U = 12
    cost = synth.cost_table(U, "flops", 0)
    n_unique = len(np.unique(cost[np.add.outer(np.arange(1, U + 1), np.arange(U)) <= U]))
    _, _, _, ev = dp_optimal_slicing(cost, 4)
    assert ev < n_unique


def test_rejects_bad_arguments():
    cost = synth.cost_table(6, "random", 0)
    with pytest.raises(ValueError):
        dp_optimal_slicing(cost, 0)
    bad = cost.copy()
    bad[0, 0] = -1
    with pytest.raises(ValueError):
        dp_optimal_slicing(bad, 2)


def test_paper_slicings_structure():
    """Printed optimal slicings sum to their sequence length in multiples of 8."""
    n = 0
    for ln in open(os.path.join(GOLD, "paper_slicings.txt")):
        if not ln.strip() or ln.startswith("#"):
            continue
        parts = ln.split()
        L = int(parts[2])
        lens = []
        for tok in parts[3:]:
            if "*" in tok:
                a, b = tok.split("*")
                lens += [int(a)] * int(b)
            else:
                lens.append(int(tok))
        assert sum(lens) == L, ln
        assert all(v % 8 == 0 for v in lens), ln
        n += 1
    assert n == 11


def test_tie_break_reading():
    """Ties are broken as documented: thresholds ascending with strict improvement,
    and within Eq. 8 the slice length k ascending with strict improvement, so among
    equal slicings the one with the shortest last slice wins.  U = 3, K = 1:
    t(1, .) = 2, t(2, .) = 2, t(3, 0) = 5; [2, 1] and [1, 2] both cost 4."""
    cost = np.full((3, 3), -7, dtype=np.int64)
    cost[0, :] = 2
    cost[1, 0] = cost[1, 1] = 2
    cost[2, 0] = 5
    units, T, tmax, _ = dp_optimal_slicing(cost, 1)
    assert T == 4 and tmax == 2
    assert units == [2, 1]
