"""Batch dimension of the slicing (Sec. 3.4): a batch of B sequences is cut into
groups of b_1 + ... + b_D = B sequences, each group pipelined with its own
optimal token slicing, the sizes minimising T_{b_1} + ... + T_{b_D}.

The oracle's knapsack is pinned to brute force over every integer partition
of B, whose enumerator is pinned to the partition numbers p(n); the C-ABI
planner must then return exactly the oracle's plan."""
import numpy as np
import pytest

from oracle import (batch_split, dp_optimal_slicing, exhaustive_batch_split, integer_partitions,
                    joint_slicing)

# p(n), the number of partitions of n (OEIS A000041), n = 1..12
PARTITION_NUMBERS = [1, 2, 3, 5, 7, 11, 15, 22, 30, 42, 56, 77]


def test_partition_enumerator_counts_and_sums():
    for n, p in enumerate(PARTITION_NUMBERS, start=1):
        parts = list(integer_partitions(n))
        assert len(parts) == p
        assert len(set(parts)) == p
        assert all(sum(q) == n and list(q) == sorted(q, reverse=True) for q in parts)


def _families(rng, B):
    yield rng.integers(1, 1000, size=B)                       # generic
    yield rng.integers(1, 4, size=B) * 10                      # many ties
    t = rng.integers(1, 1000, size=B)
    t[rng.random(B) < 0.4] = -1                                # some sizes unusable
    t[0] = max(t[0], 1)                                        # size 1 always usable
    yield t
    b = np.arange(1, B + 1)
    yield 50 + 7 * b + rng.integers(0, 5, size=B)              # per-group overhead + linear
    yield (b * 40 - b * b).clip(1)                             # concave then flat


def test_oracle_batch_split_equals_exhaustive():
    rng = np.random.default_rng(7)
    for B in range(1, 13):
        for _ in range(6):
            for T in _families(rng, B):
                T = [int(v) for v in T]
                sizes, total = batch_split(T)
                best, arg = exhaustive_batch_split(T)
                assert total == best, (T, sizes)
                assert tuple(sizes) in arg
                assert sum(sizes) == B
                assert total == sum(T[b - 1] for b in sizes)


def test_oracle_batch_split_closed_forms():
    for B in (1, 2, 5, 9):
        b = np.arange(1, B + 1)
        # a fixed cost per group: one group of all B is the unique optimum
        assert batch_split(list(100 + 3 * b)) == ([B], 100 + 3 * B)
        # superlinear cost: single sequences are the unique optimum
        assert batch_split(list(5 * b * b)) == ([1] * B, 5 * B)
        # exactly linear: every split ties; the smallest last group wins each step
        assert batch_split(list(7 * b)) == ([1] * B, 7 * B)
        # only size 1 usable
        assert batch_split([4] + [-1] * (B - 1)) == ([1] * B, 4 * B)
    # odd batch with only even sizes usable: no plan
    with pytest.raises(ValueError):
        batch_split([-1, 5, -1])


def test_oracle_joint_slicing_composes_the_two_dps():
    rng = np.random.default_rng(3)
    U, K = 6, 4
    costs = rng.integers(1, 200, size=(3, U, U)).astype(np.int64)
    groups, T_b, total = joint_slicing(costs, K)
    for b in range(3):
        assert T_b[b] == dp_optimal_slicing(costs[b], K)[1]
    assert [g[0] for g in groups] == batch_split(T_b)[0]
    assert total == sum(T_b[g[0] - 1] for g in groups)
    for b, units in groups:
        assert units == dp_optimal_slicing(costs[b - 1], K)[0]


def test_abi_batch_split_equals_oracle():
    from paper_2102_07988_amd import terapipe as tp
    rng = np.random.default_rng(11)
    for B in range(1, 13):
        for _ in range(4):
            for T in _families(rng, B):
                T = [int(v) for v in T]
                assert tp.batch_split(T) == batch_split(T), T


def test_abi_batch_split_errors():
    from paper_2102_07988_amd import terapipe as tp
    with pytest.raises(tp.TerapipeError) as e:
        tp.batch_split([-1, 5, -1])
    assert e.value.status == tp.TP_ERR_INVALID
    with pytest.raises(tp.TerapipeError):
        tp.batch_split([])


@pytest.mark.parametrize("K", [1, 3, 8])
def test_abi_joint_slicing_equals_oracle(K):
    from paper_2102_07988_amd import terapipe as tp
    rng = np.random.default_rng(100 + K)
    for B, U in ((1, 5), (2, 7), (4, 8)):
        costs = rng.integers(1, 500, size=(B, U, U)).astype(np.int64)
        # larger groups cost more per slice, less per sequence (the shape of
        # batched GEMMs): scale plane b by 0.6 b + 0.4
        for b in range(B):
            costs[b] = (costs[b] * (0.6 * (b + 1) + 0.4)).astype(np.int64)
        groups, T_b, total = tp.joint_slicing(costs, 16, K)
        og, oT, ot = joint_slicing(costs, K)
        assert T_b == oT and total == ot
        assert groups == [(b, [16 * u for u in units]) for b, units in og]
