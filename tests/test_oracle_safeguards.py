"""Oracle pins of the comparator safeguards (Sec. IV-C, Algorithm 1: for
requester-side costs the candidate set also holds the Independent, Popularity
and LocalDedup placements; comparators defined in Sec. V-A).  CPU only.

The candidates are checked against definitions written independently of the
oracle: exhaustive parent-closed optima for the per-worker profits
(Theorem 1's optimum, tie rule R1), LocalDedup's profit rebuilt from the
saving cases of Lemma 1's proof (no copy: 0; only a peer holds b:
[w - f]_+; the requester holds b: w), and objectives from Lemma 1 (Eq. 4).
"""

import numpy as np
import pytest

import oracle
from paper_2608_01655_amd import workloads as W
from tests import bruteforce as bf


def requester_instance(seed, n_max=9, m_max=3):
    """A tiny random forest with requester-side fetch costs."""
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, n_max + 1))
    m = int(rng.integers(1, m_max + 1))
    parent = W.random_forest(n, rng, p_root=float(rng.choice([0.0, 0.3])))
    lam = rng.integers(0, 6, size=(m, n)).astype(np.int64)
    w = rng.integers(0, 20, size=(m, n)).astype(np.int64)
    f_req = rng.integers(0, 25, size=(m, n)).astype(np.int64)
    f = np.zeros((m, m, n), np.int64)
    for src in range(m):
        for dst in range(m):
            if src != dst:
                f[src, dst] = f_req[dst]
    cap = rng.integers(0, n + 2, size=m).astype(np.int32)
    return parent, lam, w, f_req, f, cap


def test_requester_side_detection():
    tiny = W.make_workload("tiny")
    assert oracle.requester_side(tiny.fetch_cost)
    src_dep = W.make_workload("tree2k")
    assert not oracle.requester_side(src_dep.fetch_cost)
    _, _, _, _, f, _ = requester_instance(3, m_max=3)
    assert oracle.requester_side(f)
    if f.shape[0] >= 3:
        g = f.copy()
        g[2, 0, 0] += 1  # one source differs for requester 0
        assert not oracle.requester_side(g)
    assert oracle.requester_side(np.zeros((1, 1, 5), np.int64))  # M = 1


@pytest.mark.parametrize("seed", range(40))
def test_independent_and_popularity_are_per_worker_optima(seed):
    parent, lam, w, _, f, cap = requester_instance(seed)
    tg, _ = oracle.candidates(parent, lam, w, f, cap)
    for h in range(lam.shape[0]):
        want_i, _ = bf.best_closed_set(parent, lam[h] * w[h], int(cap[h]))
        want_p, _ = bf.best_closed_set(parent, lam[h], int(cap[h]))
        np.testing.assert_array_equal(tg[0, h], want_i)
        np.testing.assert_array_equal(tg[1, h], want_p)


def own_gain_of_local_copy(lam, w, f_req, h, b, covered):
    """Requester h's own saving on chunk b with a local copy minus without
    one, from the cases of Lemma 1's proof."""
    with_copy = w[h, b]
    without = max(w[h, b] - f_req[h, b], 0) if covered else 0
    return int(lam[h, b]) * (int(with_copy) - int(without))


@pytest.mark.parametrize("seed", range(40))
def test_localdedup_follows_the_own_saving_definition(seed):
    parent, lam, w, f_req, f, cap = requester_instance(seed)
    tg, _ = oracle.candidates(parent, lam, w, f, cap)
    m, n = lam.shape
    built = np.zeros((m, n), np.uint8)
    for h in range(m):  # workers in increasing id (reading R19)
        covered = built[:h].any(axis=0)
        p = [own_gain_of_local_copy(lam, w, f_req, h, b, bool(covered[b]))
             for b in range(n)]
        built[h], _ = bf.best_closed_set(parent, p, int(cap[h]))
    np.testing.assert_array_equal(tg[2], built)


@pytest.mark.parametrize("seed", range(25))
def test_candidate_objectives_follow_lemma1(seed):
    parent, lam, w, f_req, f, cap = requester_instance(seed)
    tg, objs = oracle.candidates(parent, lam, w, f, cap)
    for c in range(3):
        assert objs[c] == bf.requester_side_objective(lam, w, f_req, tg[c])
        assert objs[c] == oracle.objective(lam, w, f, tg[c])


@pytest.mark.parametrize("seed", range(30))
def test_plan_returns_the_argmax_with_starts_winning_ties(seed):
    parent, lam, w, _, f, cap = requester_instance(seed)
    flags = oracle.F_NO_REFINE if seed % 2 else 0
    plain = oracle.plan(parent, lam, w, f, cap, n_starts=1, flags=flags)
    sg = oracle.plan(parent, lam, w, f, cap, n_starts=1,
                     flags=flags | oracle.F_SAFEGUARDS)
    tg, objs = oracle.candidates(parent, lam, w, f, cap)
    assert sg.safeguards_run and sg.safeguard_objective == tuple(objs)
    assert sg.objective == max([plain.objective] + objs)
    assert sg.objective >= plain.objective  # never worse than the starts
    if sg.objective == plain.objective:       # ties keep the start (R20)
        assert sg.best_start == plain.best_start
        np.testing.assert_array_equal(sg.target, plain.target)
    else:
        c = sg.best_start - 1                 # S = 1
        assert objs[c] == sg.objective and all(o < sg.objective for o in objs[:c])
        np.testing.assert_array_equal(sg.target, tg[c])
    assert sg.updates == plain.updates + 3 * lam.shape[0]


def test_a_candidate_can_win():
    """The safeguard matters: some tiny requester-side instance has a
    comparator strictly above a single greedy start (no refinement)."""
    wins = 0
    for seed in range(300):
        parent, lam, w, _, f, cap = requester_instance(1000 + seed, n_max=8)
        plain = oracle.plan(parent, lam, w, f, cap, n_starts=1,
                            flags=oracle.F_NO_REFINE)
        sg = oracle.plan(parent, lam, w, f, cap, n_starts=1,
                         flags=oracle.F_NO_REFINE | oracle.F_SAFEGUARDS)
        if sg.objective > plain.objective:
            wins += 1
            assert sg.best_start >= 1
    assert wins > 0


def test_flag_is_a_no_op_for_source_dependent_costs():
    inst = W.make_workload("tree2k")
    a = oracle.plan_instance(inst, n_starts=1, max_rounds=1)
    b = oracle.plan_instance(inst, n_starts=1, max_rounds=1,
                             flags=oracle.F_SAFEGUARDS)
    assert not b.safeguards_run
    assert a.objective == b.objective and a.best_start == b.best_start
    np.testing.assert_array_equal(a.target, b.target)
