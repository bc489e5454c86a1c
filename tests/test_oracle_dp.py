"""Pins of the oracle's rooted-tree DP (Eq. 9, Theorem 1, reading R1) against
exhaustive enumeration and closed forms."""

import numpy as np
import pytest

from paper_2608_01655_amd import workloads as W
from tests import bruteforce as bf


def _closed(parent, sel):
    return all(not sel[v] or parent[v] < 0 or sel[parent[v]]
               for v in range(len(parent)))


@pytest.mark.parametrize("seed", range(400))
def test_dp_matches_bruteforce(oracle_mod, seed):
    """Theorem 1: the value is the exhaustive optimum over parent-closed sets
    of size <= k; under R1 the set is the lexicographically smallest optimal
    0/1 vector in canonical preorder (many ties: profits in {0,1,2})."""
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 13))
    parent = W.random_forest(n, rng)
    profit = rng.integers(0, 3, size=n).astype(np.int64)
    k = int(rng.integers(0, n + 2))
    sel, val = oracle_mod.rooted_dp(parent, profit, k)
    bsel, bval = bf.best_closed_set(parent, profit, k)
    assert val == bval
    np.testing.assert_array_equal(sel, bsel)


@pytest.mark.parametrize("seed", range(60))
def test_dp_matches_bruteforce_wide_values(oracle_mod, seed):
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(6, 13))
    parent = W.random_forest(n, rng, p_root=0.3)
    profit = rng.integers(0, 10 ** 12, size=n).astype(np.int64)
    profit[rng.random(n) < 0.3] = 0
    k = int(rng.integers(1, n + 1))
    sel, val = oracle_mod.rooted_dp(parent, profit, k)
    bsel, bval = bf.best_closed_set(parent, profit, k)
    assert val == bval
    np.testing.assert_array_equal(sel, bsel)


def test_path_tree_is_best_shortest_prefix(oracle_mod):
    """On a path the feasible sets are prefixes: the answer is the shortest
    prefix of length <= k with the largest sum."""
    rng = np.random.default_rng(7)
    for trial in range(50):
        n = int(rng.integers(1, 40))
        parent = np.arange(-1, n - 1, dtype=np.int32)
        profit = rng.integers(0, 5, size=n).astype(np.int64)
        k = int(rng.integers(0, n + 3))
        sums = np.concatenate([[0], np.cumsum(profit)])
        L = int(np.argmax(sums[: min(k, n) + 1]))  # first maximiser = shortest
        sel, val = oracle_mod.rooted_dp(parent, profit, k)
        assert val == int(sums[L])
        assert sel.tolist() == [1] * L + [0] * (n - L)


def test_star_takes_root_and_top_leaves(oracle_mod):
    """Root plus leaves with distinct positive profits: for k >= 1 the
    answer is the root and the k-1 most profitable leaves."""
    rng = np.random.default_rng(3)
    for trial in range(30):
        leaves = int(rng.integers(1, 30))
        n = leaves + 1
        parent = np.array([-1] + [0] * leaves, dtype=np.int32)
        profit = np.concatenate([[int(rng.integers(1, 100))],
                                 rng.permutation(leaves) * 3 + 1]).astype(np.int64)
        k = int(rng.integers(1, n + 2))
        sel, val = oracle_mod.rooted_dp(parent, profit, k)
        top = np.sort(profit[1:])[::-1][: min(k, n) - 1]
        assert val == int(profit[0] + top.sum())
        assert sel[0] == 1 and sel.sum() == min(k, n)


def test_zero_budget_and_zero_profit_give_empty(oracle_mod):
    rng = np.random.default_rng(11)
    parent = W.random_forest(30, rng)
    profit = rng.integers(1, 9, size=30).astype(np.int64)
    sel, val = oracle_mod.rooted_dp(parent, profit, 0)
    assert val == 0 and sel.sum() == 0
    sel, val = oracle_mod.rooted_dp(parent, np.zeros(30, np.int64), 30)
    assert val == 0 and sel.sum() == 0


def test_unbounded_budget_takes_every_positive_closure(oracle_mod):
    """k >= n: with all profits positive every node is taken."""
    rng = np.random.default_rng(5)
    parent = W.random_forest(50, rng)
    profit = rng.integers(1, 9, size=50).astype(np.int64)
    for k in (50, 51, 10 ** 6):
        sel, val = oracle_mod.rooted_dp(parent, profit, k)
        assert sel.sum() == 50 and val == int(profit.sum())


def test_dp_invariants_at_size(oracle_mod):
    """On larger random trees: selection is parent-closed, within budget, its
    profit equals the value, and the value is nondecreasing in k."""
    rng = np.random.default_rng(21)
    n = 3000
    parent = W.random_forest(n, rng, p_root=0.02)
    profit = rng.integers(0, 1000, size=n).astype(np.int64)
    last = -1
    for k in (0, 1, 2, 17, 64, 65, 300, 1000, n, n + 5):
        sel, val = oracle_mod.rooted_dp(parent, profit, k)
        assert _closed(parent, sel)
        assert sel.sum() <= k
        assert int(profit[sel.astype(bool)].sum()) == val
        assert val >= last
        last = val


def test_preorder_and_next(oracle_mod):
    rng = np.random.default_rng(2)
    for _ in range(30):
        n = int(rng.integers(1, 60))
        parent = W.random_forest(n, rng)
        order, nxt = oracle_mod.preorder(parent)
        assert order.tolist() == bf.canonical_preorder(parent)
        pos = np.empty(n, np.int64)
        pos[order] = np.arange(n)
        # next(i) - i is the subtree size
        size = np.ones(n, np.int64)
        for v in order[::-1]:
            if parent[v] >= 0:
                size[parent[v]] += size[v]
        assert np.all(nxt == np.arange(n) + size[order])


def test_invalid_trees_rejected(oracle_mod):
    with pytest.raises(oracle_mod.OracleError) as e:
        oracle_mod.rooted_dp(np.array([1, 0], np.int32), np.ones(2, np.int64), 1)
    assert e.value.code == oracle_mod.E_TREE
    with pytest.raises(oracle_mod.OracleError) as e:
        oracle_mod.rooted_dp(np.array([-1, 5], np.int32), np.ones(2, np.int64), 1)
    assert e.value.code == oracle_mod.E_TREE
    with pytest.raises(oracle_mod.OracleError) as e:
        oracle_mod.rooted_dp(np.array([-1, 1], np.int32), np.ones(2, np.int64), 1)
    assert e.value.code == oracle_mod.E_TREE
    with pytest.raises(oracle_mod.OracleError) as e:
        oracle_mod.rooted_dp(np.array([-1, 0], np.int32), np.array([1, -1]), 1)
    assert e.value.code == oracle_mod.E_RANGE
