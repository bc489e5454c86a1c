"""Pins of the oracle's whole planner (Algorithm 1) against Theorem 3's
1/2 bound with exhaustive optima, the monotonicity of coordinate refinement
(Sec. IV-C), closed-form special cases and Theorem 2's spider construction,
plus the start orders (readings R6-R8) and SplitMix64's published outputs."""

import itertools
import math

import numpy as np
import pytest

from paper_2608_01655_amd import workloads as W
from tests import bruteforce as bf


def _closed(parent, sel):
    return all(not sel[v] or parent[v] < 0 or sel[parent[v]]
               for v in range(len(parent)))


def _feasible(inst, tgt):
    for h in range(inst.m):
        assert tgt[h].sum() <= inst.cap[h]
        assert _closed(inst.parent, tgt[h])


@pytest.mark.parametrize("seed", range(25))
def test_theorem3_half_bound_and_refinement(oracle_mod, seed):
    """Every fixed-order greedy start reaches >= 1/2 of the exhaustive OPT
    (Theorem 3); refinement never lowers a start's value (Sec. IV-C)."""
    rng = np.random.default_rng(seed)
    m = int(rng.integers(2, 4))
    n = int(rng.integers(3, 7))
    inst = W.random_instance(n, m, rng, kmax=3,
                             source_dependent=bool(seed % 2))
    opt = bf.joint_optimum(inst.parent, inst.demand, inst.recompute_cost,
                           inst.fetch_cost, inst.cap)
    orders = np.array(list(itertools.permutations(range(m))), np.int32)
    greedy = oracle_mod.plan_instance(inst, n_starts=len(orders),
                                      orders_in=orders,
                                      flags=oracle_mod.F_NO_REFINE)
    refined = oracle_mod.plan_instance(inst, n_starts=len(orders),
                                       orders_in=orders)
    assert np.all(2 * greedy.start_objective >= opt)
    assert np.all(refined.start_objective >= greedy.start_objective)
    assert np.all(refined.start_objective <= opt)
    assert refined.objective == refined.start_objective.max()
    assert np.all(greedy.start_sweeps == 0)
    assert np.all(refined.start_sweeps >= 1)
    _feasible(inst, refined.target)
    # the returned objective is the objective of the returned placement
    assert refined.objective == oracle_mod.objective(
        inst.demand, inst.recompute_cost, inst.fetch_cost, refined.target)


def test_refinement_accepts_strictly_improve(oracle_mod):
    """Each accepted replacement raises G strictly, so a start with a accepts
    ends strictly above its greedy value, and one with none ends equal."""
    rng = np.random.default_rng(77)
    seen_accept = False
    for trial in range(40):
        inst = W.random_instance(int(rng.integers(8, 30)),
                                 int(rng.integers(2, 5)), rng, kmax=8)
        g = oracle_mod.plan_instance(inst, n_starts=3,
                                     flags=oracle_mod.F_NO_REFINE)
        r = oracle_mod.plan_instance(inst, n_starts=3)
        for s in range(3):
            if r.start_accepts[s] > 0:
                seen_accept = True
                assert r.start_objective[s] > g.start_objective[s]
            else:
                assert r.start_objective[s] == g.start_objective[s]
                assert r.start_sweeps[s] == 1
    assert seen_accept


def test_single_worker_is_one_exact_dp(oracle_mod):
    """M = 1: the plan is one rooted-tree solve with p = Lambda * w."""
    rng = np.random.default_rng(4)
    for _ in range(20):
        inst = W.random_instance(int(rng.integers(1, 40)), 1, rng)
        res = oracle_mod.plan_instance(inst, n_starts=2)
        sel, val = oracle_mod.rooted_dp(inst.parent,
                                        inst.demand[0] * inst.recompute_cost[0],
                                        int(inst.cap[0]))
        assert res.objective == val
        assert np.array_equal(res.target[0], sel)


def test_fetch_never_cheaper_means_independent_workers(oracle_mod):
    """f >= w everywhere: Delta = 0 (Eq. 3), so each worker's plan is its own
    DP with p = Lambda_m * w_m, identical for every start, with no accepted
    refinement (Sec. III-B)."""
    rng = np.random.default_rng(8)
    for _ in range(10):
        m = int(rng.integers(2, 5))
        inst = W.random_instance(int(rng.integers(5, 40)), m, rng)
        inst.fetch_cost = inst.fetch_cost + 10 ** 6
        res = oracle_mod.plan_instance(inst, n_starts=4)
        assert np.all(res.start_accepts == 0)
        assert np.all(res.start_sweeps == 1)
        assert np.all(res.start_objective == res.objective)
        total = 0
        for h in range(m):
            sel, val = oracle_mod.rooted_dp(
                inst.parent, inst.demand[h] * inst.recompute_cost[h],
                int(inst.cap[h]))
            assert np.array_equal(res.target[h], sel)
            total += val
        assert res.objective == total


def _spider(sizes, q, B):
    """Theorem 2's reduction: legs of s_i chunks under the dummy root, q
    holders of budget B and one requester of budget 0, w(d) = 2d, f = 1,
    requester demand L/s_i on leg i (L = lcm of the s_i)."""
    L = math.lcm(*sizes)
    parent, depth, lamr = [], [], []
    for s in sizes:
        for d in range(1, s + 1):
            parent.append(-1 if d == 1 else len(parent) - 1)
            depth.append(d)
            lamr.append(L // s)
    n, m = len(parent), q + 1
    lam = np.zeros((m, n), np.int64)
    lam[q] = lamr
    w = np.tile(2 * np.array(depth, np.int64), (m, 1))
    f = np.ones((m, m, n), np.int64)
    cap = np.array([B] * q + [0], np.int32)
    return np.array(parent, np.int32), lam, w, f, cap, L


def test_theorem2_spider_single_holder(oracle_mod):
    """q = 1, s = (4,4,4), B = 12: the holder can cover every leg, reaching
    L*q*B; covering x_i chunks of leg i saves L*x_i^2/s_i."""
    parent, lam, w, f, cap, L = _spider((4, 4, 4), 1, 12)
    res = oracle_mod.plan(parent, lam, w, f, cap, n_starts=2)
    assert res.objective == L * 12
    assert res.target[0].sum() == 12 and res.target[1].sum() == 0


def test_theorem2_spider_with_partition(oracle_mod):
    """q = 2, B = 20, s = (6,7,7,6,7,7) has a 3-partition: OPT = L*q*B and the
    plan is within [OPT/2, OPT] (Theorems 2 and 3)."""
    parent, lam, w, f, cap, L = _spider((6, 7, 7, 6, 7, 7), 2, 20)
    res = oracle_mod.plan(parent, lam, w, f, cap, n_starts=0)
    assert L * 20 <= res.objective <= L * 40
    # the saving is exactly sum_i L * x_i^2 / s_i over covered leg prefixes
    covered = res.target[:2].max(axis=0)
    start, tot = 0, 0
    for s in (6, 7, 7, 6, 7, 7):
        x = int(covered[start: start + s].sum())
        assert covered[start: start + x].all()
        tot += L * x * x // s
        start += s
    assert tot == res.objective


def test_theorem2_spider_without_partition(oracle_mod):
    """s = (6,6,6,6,7,9), B = 20 admits no 3-partition, so no placement can
    reach L*q*B."""
    parent, lam, w, f, cap, L = _spider((6, 6, 6, 6, 7, 9), 2, 20)
    res = oracle_mod.plan(parent, lam, w, f, cap, n_starts=0)
    assert L * 20 <= res.objective < L * 40


def test_splitmix64_published_outputs(oracle_mod):
    """SplitMix64 seeded with 1234567: the first five outputs as published
    with the generator's reference description."""
    assert oracle_mod.splitmix64_stream(1234567, 5) == [
        6457827717110365317, 3203168211198807973, 9817491932198370423,
        4593380528125082431, 16408922859458223821]


def test_orders_readings(oracle_mod):
    st = np.array([5, 9, 5], np.int64)
    o = oracle_mod.orders(3, 2, 0, st)
    assert o.tolist() == [[1, 0, 2], [2, 0, 1]]
    o = oracle_mod.orders(3, 0, 0, st)  # paper default for M <= 5
    assert o.tolist() == [list(p) for p in itertools.permutations(range(3))]
    o = oracle_mod.orders(7, 0, 3, np.arange(7))
    assert o.shape == (8, 7)
    assert o[0].tolist() == [6, 5, 4, 3, 2, 1, 0]
    assert o[1].tolist() == list(range(7))
    for row in o:
        assert sorted(row.tolist()) == list(range(7))
    # start s >= 2 is a Fisher-Yates shuffle driven by SplitMix64(seed + s)
    for s in range(2, 8):
        x = oracle_mod.splitmix64_stream(3 + s, 6)
        perm = list(range(7))
        for t, i in enumerate(range(6, 0, -1)):
            j = x[t] % (i + 1)
            perm[i], perm[j] = perm[j], perm[i]
        assert o[s].tolist() == perm


def test_plan_statistics_and_capacity_cap(oracle_mod):
    rng = np.random.default_rng(12)
    inst = W.random_instance(20, 3, rng, kmax=40)
    res = oracle_mod.plan_instance(inst, n_starts=3, max_rounds=2)
    assert np.all(res.start_sweeps <= 2)
    cells_pass = sum(20 * min(int(k), 20) for k in inst.cap)
    assert res.updates == 3 + sum(3 * (1 + int(r)) for r in res.start_sweeps)
    assert res.dp_cells == cells_pass * (1 + sum(1 + int(r) for r in res.start_sweeps))
    _feasible(inst, res.target)


def test_plan_rejects_bad_input(oracle_mod):
    rng = np.random.default_rng(1)
    inst = W.random_instance(6, 2, rng)
    with pytest.raises(oracle_mod.OracleError) as e:
        oracle_mod.plan(np.array([1, 2, 0, -1, -1, -1], np.int32), inst.demand,
                        inst.recompute_cost, inst.fetch_cost, inst.cap)
    assert e.value.code == oracle_mod.E_TREE
    with pytest.raises(oracle_mod.OracleError) as e:
        oracle_mod.plan(inst.parent, inst.demand, inst.recompute_cost,
                        inst.fetch_cost, np.array([1, -1], np.int32))
    assert e.value.code == oracle_mod.E_RANGE
    with pytest.raises(oracle_mod.OracleError) as e:
        oracle_mod.plan_instance(inst, n_starts=1,
                                 orders_in=np.array([[0, 0]], np.int32))
    assert e.value.code == oracle_mod.E_ARG


def test_start_ties_go_to_earliest(oracle_mod):
    """R10: two identical workers planned in mirrored orders reach the same
    objective with mirrored placements; the earliest start must be returned."""
    rng = np.random.default_rng(31)
    n = 12
    parent = W.random_forest(n, rng, shuffle=False)
    lam1 = rng.integers(1, 50, size=n)
    w1 = rng.integers(10, 100, size=n)
    lam = np.stack([lam1, lam1]).astype(np.int64)
    w = np.stack([w1, w1]).astype(np.int64)
    f = np.ones((2, 2, n), np.int64)  # remote copies almost as good as local
    cap = np.array([3, 3], np.int32)
    both = oracle_mod.plan(parent, lam, w, f, cap, n_starts=2,
                           orders_in=np.array([[0, 1], [1, 0]], np.int32))
    assert both.start_objective[0] == both.start_objective[1]
    first = oracle_mod.plan(parent, lam, w, f, cap, n_starts=1,
                            orders_in=np.array([[0, 1]], np.int32))
    second = oracle_mod.plan(parent, lam, w, f, cap, n_starts=1,
                             orders_in=np.array([[1, 0]], np.int32))
    assert not np.array_equal(first.target, second.target)
    assert both.best_start == 0
    assert np.array_equal(both.target, first.target)
