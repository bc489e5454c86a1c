"""Pins of the oracle's objective (Eq. 6) and marginal (Eq. 7) against the
paper's structural results: Lemma 1 (requester-side modular-plus-coverage
form), Proposition 1 (exact additive marginal), Eq. (10), monotonicity and
submodularity."""

import numpy as np
import pytest

from paper_2608_01655_amd import workloads as W
from tests import bruteforce as bf


def _rand_target(rng, m, n, p=0.4):
    return (rng.random((m, n)) < p).astype(np.uint8)


@pytest.mark.parametrize("seed", range(40))
def test_lemma1_decomposition(oracle_mod, seed):
    """With source-independent fetch costs (R12: rows equal over src), F_pair
    equals Lemma 1's sum of local values plus first-replica coverage."""
    rng = np.random.default_rng(seed)
    m = int(rng.integers(1, 6))
    n = int(rng.integers(1, 25))
    inst = W.random_instance(n, m, rng, source_dependent=False)
    # requester-side cost of requester r: any off-diagonal source row
    f_req = np.array([inst.fetch_cost[(r + 1) % m, r] for r in range(m)])
    tgt = _rand_target(rng, m, n)
    got = oracle_mod.objective(inst.demand, inst.recompute_cost,
                               inst.fetch_cost, tgt)
    want = bf.requester_side_objective(inst.demand, inst.recompute_cost,
                                       f_req, tgt)
    assert got == want


@pytest.mark.parametrize("seed", range(40))
def test_eq10_requester_side_marginal(oracle_mod, seed):
    rng = np.random.default_rng(100 + seed)
    m = int(rng.integers(1, 6))
    n = int(rng.integers(1, 25))
    inst = W.random_instance(n, m, rng, source_dependent=False)
    f_req = np.array([inst.fetch_cost[(r + 1) % m if m > 1 else 0, r]
                      for r in range(m)])
    tgt = _rand_target(rng, m, n)
    h = int(rng.integers(0, m))
    prof, _ = oracle_mod.marginal(inst.demand, inst.recompute_cost,
                                  inst.fetch_cost, tgt, h)
    want = bf.requester_side_marginal(inst.demand, inst.recompute_cost, f_req,
                                      tgt, h)
    assert prof.tolist() == want


@pytest.mark.parametrize("seed", range(60))
def test_prop1_marginal_is_exact_gain(oracle_mod, seed):
    """Proposition 1: for any S, G(T_-h with h holding S) - G(T_-h) equals
    the sum of p_h over S, and g_without_h = G(T_-h)."""
    rng = np.random.default_rng(200 + seed)
    m = int(rng.integers(1, 6))
    n = int(rng.integers(1, 30))
    inst = W.random_instance(n, m, rng, source_dependent=True)
    tgt = _rand_target(rng, m, n)
    h = int(rng.integers(0, m))
    prof, g_wo = oracle_mod.marginal(inst.demand, inst.recompute_cost,
                                     inst.fetch_cost, tgt, h)
    t0 = tgt.copy()
    t0[h] = 0
    g0 = oracle_mod.objective(inst.demand, inst.recompute_cost,
                              inst.fetch_cost, t0)
    assert g_wo == g0
    for _ in range(5):
        S = (rng.random(n) < 0.5).astype(np.uint8)
        t1 = t0.copy()
        t1[h] = S
        g1 = oracle_mod.objective(inst.demand, inst.recompute_cost,
                                  inst.fetch_cost, t1)
        assert g1 - g0 == int(prof[S.astype(bool)].sum())


def test_single_holder_closed_form(oracle_mod):
    """One holder h of chunk b: requester m saves Lambda_m(b) * q_{m<-h}(b);
    the holder itself saves Lambda_h(b) * w_h(b) (Eq. 5)."""
    lam = np.array([[3, 0], [5, 7]], np.int64)
    w = np.array([[100, 10], [40, 90]], np.int64)
    f = np.zeros((2, 2, 2), np.int64)
    f[0, 1] = [15, 200]  # requester 1 fetching from holder 0
    f[1, 0] = [30, 1]
    tgt = np.array([[1, 1], [0, 0]], np.uint8)
    # requester 0 holds both: 3*100 + 0*10; requester 1 fetches from 0:
    # b0: 5*(40-15) = 125; b1: 7*max(90-200, 0) = 0
    assert oracle_mod.objective(lam, w, f, tgt) == 300 + 125
    tgt = np.array([[0, 0], [1, 0]], np.uint8)
    # requester 1 holds b0: 5*40; requester 0 fetches b0 from 1: 3*(100-30)
    assert oracle_mod.objective(lam, w, f, tgt) == 200 + 210


@pytest.mark.parametrize("seed", range(20))
def test_monotone_submodular(oracle_mod, seed):
    """Lemma 1 / Proposition 1: G is monotone and has diminishing returns
    over worker-chunk elements."""
    rng = np.random.default_rng(300 + seed)
    m = int(rng.integers(2, 5))
    n = int(rng.integers(2, 15))
    inst = W.random_instance(n, m, rng, source_dependent=True)
    G = lambda t: oracle_mod.objective(inst.demand, inst.recompute_cost,
                                       inst.fetch_cost, t)
    elems = [(h, b) for h in range(m) for b in range(n)]
    rng.shuffle(elems)
    A = np.zeros((m, n), np.uint8)
    for cut in range(0, len(elems) - 1, 3):
        B = A.copy()
        for (h, b) in elems[cut: cut + 3]:
            B[h, b] = 1
        e = elems[-1]
        if B[e] or A[e]:
            continue
        gA, gB = G(A), G(B)
        assert gB >= gA
        Ae, Be = A.copy(), B.copy()
        Ae[e] = 1
        Be[e] = 1
        assert G(Ae) - gA >= G(Be) - gB
        A = B


def test_fetch_diagonal_ignored(oracle_mod):
    """R11: fetch_cost[h][h][*] plays no part."""
    rng = np.random.default_rng(9)
    inst = W.random_instance(12, 3, rng)
    tgt = _rand_target(rng, 3, 12)
    f2 = inst.fetch_cost.copy()
    for h in range(3):
        f2[h, h] = rng.integers(0, 1000, size=12)
    a = oracle_mod.objective(inst.demand, inst.recompute_cost, inst.fetch_cost, tgt)
    b = oracle_mod.objective(inst.demand, inst.recompute_cost, f2, tgt)
    assert a == b
    pa, ga = oracle_mod.marginal(inst.demand, inst.recompute_cost, inst.fetch_cost, tgt, 1)
    pb, gb = oracle_mod.marginal(inst.demand, inst.recompute_cost, f2, tgt, 1)
    assert ga == gb and np.array_equal(pa, pb)


def test_value_errors(oracle_mod):
    lam = np.ones((2, 3), np.int64)
    w = np.ones((2, 3), np.int64)
    f = np.ones((2, 2, 3), np.int64)
    t = np.zeros((2, 3), np.uint8)
    bad = w.copy()
    bad[1, 2] = -1
    with pytest.raises(oracle_mod.OracleError) as e:
        oracle_mod.objective(lam, bad, f, t)
    assert e.value.code == oracle_mod.E_RANGE
    big = np.full((2, 3), 2 ** 31, np.int64)
    with pytest.raises(oracle_mod.OracleError) as e:
        oracle_mod.objective(big, big, f, t)
    assert e.value.code == oracle_mod.E_OVERFLOW
