"""GPU parity of the per-update entry points against the CPU oracle:
pp_rooted_dp (Eq. 9 sweep + backtrack), pp_marginal (Eq. 7) and
pp_objective (Eq. 6).  Integer work, so every comparison is bit-exact."""

import os

import numpy as np
import pytest

from paper_2608_01655_amd import binding as B
from paper_2608_01655_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _say_case(request):
    print(f"\n[case] {request.node.name}", flush=True)
    yield


def _dp_case(oracle_mod, parent, profit, k):
    sel, val = B.pp_rooted_dp(parent, profit, k)
    osel, oval = oracle_mod.rooted_dp(parent, profit, k)
    assert val == oval
    np.testing.assert_array_equal(sel, osel)


@pytest.mark.parametrize("seed", range(60))
def test_rooted_dp_random(oracle_mod, seed):
    """Random forests with shuffled labels, tie-heavy profits, budgets that
    cross 64-cell stage boundaries and exceed n."""
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 400))
    parent = W.random_forest(n, rng, p_root=float(rng.choice([0.0, 0.05, 0.3])))
    hi = int(rng.choice([2, 5, 1000, 10 ** 9]))
    profit = rng.integers(0, hi, size=n).astype(np.int64)
    k = int(rng.choice([1, 2, 63, 64, 65, 127, 128, 129, 200, n, n + 7,
                        int(rng.integers(0, n + 2))]))
    _dp_case(oracle_mod, parent, profit, k)


@pytest.mark.parametrize("cells", [1, 2, 4])
def test_rooted_dp_each_lane_width(oracle_mod, cells, monkeypatch):
    """Every compiled cells-per-lane variant of the sweep (1, 2 and 4 cells
    per lane, forced through PP_DP_CELLS)."""
    monkeypatch.setenv("PP_DP_CELLS", str(cells))
    rng = np.random.default_rng(100 + cells)
    for n, k in ((1, 1), (70, 69), (3000, 1000), (2500, 2500)):
        parent = W.random_forest(n, rng, p_root=0.02)
        profit = rng.integers(0, 50, size=n).astype(np.int64)
        _dp_case(oracle_mod, parent, profit, k)


def test_rooted_dp_shapes(oracle_mod):
    """Degenerate trees: a path, a star, a comb whose spine comes first (a
    deep stack of pending skip rows), a forest of singletons."""
    rng = np.random.default_rng(7)
    n = 1500
    path = np.arange(-1, n - 1, dtype=np.int32)
    star = np.array([-1] + [0] * (n - 1), np.int32)
    # spine 0..199 with a leaf 200+d under spine node d: the spine child has
    # the smaller id, so every leaf's row is a far skip target (depth 200)
    comb = np.array([-1] + list(range(0, 199)) + list(range(0, 200)), np.int32)
    flat = np.full(n, -1, np.int32)
    for parent in (path, star, comb, flat):
        nn = parent.shape[0]
        profit = rng.integers(0, 100, size=nn).astype(np.int64)
        for k in (0, 1, 64, 65, 777, nn):
            _dp_case(oracle_mod, parent, profit, k)


@pytest.mark.parametrize("n", [511, 512, 513, 1023, 1024, 1025, 1553, 2065])
def test_rooted_dp_super_window_edges(oracle_mod, n):
    """The backtrack stages rows in blocks of 512 (16 windows of 32): sizes
    at and around those boundaries, sparse profits so that the walk skips
    whole subtrees across window and block boundaries, and budgets that end
    the walk inside a block, at a stage edge or past the last row."""
    rng = np.random.default_rng(5000 + n)
    for p_root in (0.0, 0.01, 0.2):
        parent = W.random_forest(n, rng, p_root=p_root)
        for density in (0.05, 0.5):
            profit = (rng.integers(1, 1000, size=n) *
                      (rng.random(n) < density)).astype(np.int64)
            for k in (64, 65, 300, n // 2, n, n + 1):
                _dp_case(oracle_mod, parent, profit, k)


def test_rooted_dp_all_zero_and_huge(oracle_mod):
    rng = np.random.default_rng(3)
    parent = W.random_forest(500, rng)
    _dp_case(oracle_mod, parent, np.zeros(500, np.int64), 300)
    big = np.full(500, (2 ** 63 - 1) // 500, np.int64)
    _dp_case(oracle_mod, parent, big, 499)


@pytest.mark.parametrize("name,k", [("tree50k", 4096), ("chat50k", 8192)])
def test_rooted_dp_full_size(oracle_mod, name, k):
    """The benchmark trees at their full capacity, with demand-weighted
    profits (the standalone marginal of worker 0)."""
    inst = W.make_workload(name)
    profit = inst.demand[0] * inst.recompute_cost[0]
    _dp_case(oracle_mod, inst.parent, profit, k)


@pytest.mark.parametrize("seed", range(30))
def test_marginal_and_objective(oracle_mod, seed):
    rng = np.random.default_rng(500 + seed)
    m = int(rng.integers(1, 7))
    n = int(rng.integers(1, 500))
    inst = W.random_instance(n, m, rng, source_dependent=bool(seed % 3),
                             value_range=int(rng.choice([4, 100, 10 ** 6])))
    tgt = (rng.random((m, n)) < rng.random()).astype(np.uint8)
    for h in range(m):
        p, g = B.pp_marginal(inst.demand, inst.recompute_cost, inst.fetch_cost,
                             tgt, h)
        op, og = oracle_mod.marginal(inst.demand, inst.recompute_cost,
                                     inst.fetch_cost, tgt, h)
        np.testing.assert_array_equal(p, op)
        assert g == og
    assert B.pp_objective(inst.demand, inst.recompute_cost, inst.fetch_cost,
                          tgt) == oracle_mod.objective(
        inst.demand, inst.recompute_cost, inst.fetch_cost, tgt)


def test_errors_on_gpu_entry_points():
    with pytest.raises(B.PPError) as e:
        B.pp_rooted_dp(np.array([-1, 0], np.int32), np.array([1, -2]), 1)
    assert e.value.code == B.PP_E_RANGE
    with pytest.raises(B.PPError) as e:
        B.pp_marginal(np.ones((2, 3)), np.ones((2, 3)), np.ones((2, 2, 3)),
                      np.zeros((2, 3)), 2)
    assert e.value.code == B.PP_E_ARG
