"""GPU parity of epoch re-planning (Sec. IV-D: plan the refreshed inputs,
evaluate the incumbent under them, adopt only if the horizon's saving exceeds
the one-time materialization cost) against the CPU oracle: decision, both
objectives, the one-time cost, the proposal and the returned target --
bit-exact."""

import hashlib
import json
import os

import numpy as np
import pytest

from paper_2608_01655_amd import binding as B
from paper_2608_01655_amd import workloads as W

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "replans.json")


@pytest.fixture(autouse=True)
def _say_case(request):
    print(f"\n[case] {request.node.name}", flush=True)
    yield


def _same(g, o):
    assert g.adopt == o.adopt
    assert g.incumbent_objective == o.incumbent_objective
    assert g.proposal_objective == o.proposal_objective
    assert g.materialization_cost == o.materialization_cost
    np.testing.assert_array_equal(g.proposal, o.proposal)
    np.testing.assert_array_equal(g.target, o.target)


def _both(oracle_mod, parent, lam, w, f, cap, inc, horizon, **kw):
    kw = dict(dict(n_starts=1, max_rounds=0, order_seed=0), **kw)
    g = B.pp_replan(parent, lam, w, f, cap, inc, horizon, **kw)
    o = oracle_mod.replan(parent, lam, w, f, cap, inc, horizon, threads=8, **kw)
    return g, o


@pytest.mark.parametrize("seed", range(30))
def test_replan_random(oracle_mod, seed):
    rng = np.random.default_rng(700 + seed)
    m = int(rng.integers(1, 6))
    n = int(rng.integers(1, 260))
    inst = W.random_instance(n, m, rng, kmax=int(rng.choice([3, 40, n + 2])),
                             source_dependent=bool(seed % 3),
                             value_range=int(rng.choice([5, 100, 10 ** 5])))
    # incumbents need not be parent-closed or within the new capacities
    inc = (rng.random((m, n)) < rng.choice([0.0, 0.1, 0.5, 1.0])).astype(np.uint8)
    horizon = int(rng.choice([0, 1, 7, 1000, 10 ** 12]))
    flags = (B.PP_F_NO_REFINE if seed % 2 else 0) | \
        (B.PP_F_SAFEGUARDS if seed % 3 == 0 else 0)
    g, o = _both(oracle_mod, inst.parent, inst.demand, inst.recompute_cost,
                 inst.fetch_cost, inst.cap, inc, horizon,
                 n_starts=int(rng.integers(0, 4)),
                 max_rounds=int(rng.integers(0, 3)),
                 order_seed=int(rng.integers(0, 2 ** 62)), flags=flags)
    _same(g, o)
    assert g.plan.objective == o.proposal_objective


@pytest.mark.parametrize("shift", [(1, 4), (1, 2), (1, 1), "sigma0.5", "sigma1.0"])
def test_replan_demand_shift_tree2k(oracle_mod, shift):
    """The paper's transition kinds on the 2,000-chunk tree: a 25/50/100%
    routing shift or a log-normal popularity perturbation; the incumbent is
    the oracle's plan of the previous epoch."""
    inst = W.make_workload("tree2k")
    kw = dict(n_starts=inst.n_starts, max_rounds=inst.max_rounds,
              order_seed=inst.order_seed)
    old = oracle_mod.plan_instance(inst, threads=8)
    if isinstance(shift, tuple):
        lam = W.shift_routing(inst.parent, inst.demand, *shift)
    else:
        lam = W.perturb_popularity(inst.parent, inst.demand, float(shift[5:]),
                                   np.random.default_rng(21))
    for horizon in (1, 100, 10 ** 6):
        g, o = _both(oracle_mod, inst.parent, lam, inst.recompute_cost,
                     inst.fetch_cost, inst.cap, old.target, horizon, **kw)
        _same(g, o)


def test_replan_rag10k_full_shift(oracle_mod):
    """The 10,000-chunk RAG-shaped tree, 8 workers, every request routed to
    the next worker; the incumbent is the oracle's previous-epoch plan."""
    inst = W.make_workload("rag10k")
    kw = dict(n_starts=inst.n_starts, max_rounds=inst.max_rounds,
              order_seed=inst.order_seed)
    old = oracle_mod.plan_instance(inst, threads=8)
    lam = W.shift_routing(inst.parent, inst.demand, 1, 1)
    g, o = _both(oracle_mod, inst.parent, lam, inst.recompute_cost,
                 inst.fetch_cost, inst.cap, old.target, 50, **kw)
    _same(g, o)
    assert g.materialization_cost > 0


def test_replan_incumbent_equal_to_the_plan(oracle_mod):
    inst = W.make_workload("tree2k")
    kw = dict(n_starts=1, max_rounds=1, order_seed=inst.order_seed)
    cur = oracle_mod.plan_instance(inst, threads=8, **kw)
    g, o = _both(oracle_mod, inst.parent, inst.demand, inst.recompute_cost,
                 inst.fetch_cost, inst.cap, cur.target, 10 ** 9, **kw)
    _same(g, o)
    assert g.materialization_cost == 0 and not g.adopt


def test_replan_equality_and_huge_horizon(oracle_mod):
    parent = np.array([-1], np.int32)
    lam = np.array([[1]], np.int64)
    w = np.array([[10]], np.int64)
    f = np.zeros((1, 1, 1), np.int64)
    cap = np.array([1], np.int32)
    inc = np.zeros((1, 1), np.uint8)
    for horizon, adopt in ((0, False), (1, False), (2, True)):
        g, o = _both(oracle_mod, parent, lam, w, f, cap, inc, horizon)
        _same(g, o)
        assert g.adopt == adopt
    inst = W.make_workload("tiny")
    z = np.zeros((inst.m, inst.n), np.uint8)
    g, o = _both(oracle_mod, inst.parent, inst.demand, inst.recompute_cost,
                 inst.fetch_cost, inst.cap, z, 2 ** 62)
    _same(g, o)
    assert g.adopt  # the product exceeds INT64_MAX and must not wrap


def test_replan_tree50k_golden():
    """The 50,000-chunk, 16-worker tree after a 50% routing shift, at the
    benchmark's start settings, against the oracle's stored decision."""
    with open(GOLDEN) as fh:
        gold = json.load(fh)["tree50k-shift50"]
    inst = W.make_workload("tree50k")
    lam = W.shift_routing(inst.parent, inst.demand, *gold["shift"])
    assert hashlib.sha256(lam.tobytes()).hexdigest() == gold["demand_sha256"]
    inc = W.prefix_incumbent(inst.n, inst.cap)
    g = B.pp_replan(inst.parent, lam, inst.recompute_cost, inst.fetch_cost,
                    inst.cap, inc, gold["horizon"], n_starts=inst.n_starts,
                    max_rounds=inst.max_rounds, order_seed=inst.order_seed)
    assert g.adopt == gold["adopt"]
    assert g.incumbent_objective == gold["incumbent_objective"]
    assert g.proposal_objective == gold["proposal_objective"]
    assert g.materialization_cost == gold["materialization_cost"]
    rows = [hashlib.sha256(g.proposal[h].tobytes()).hexdigest()
            for h in range(inst.m)]
    assert rows == gold["proposal_row_sha256"]
    np.testing.assert_array_equal(g.target, g.proposal if g.adopt else inc)


# ---------------------------------------------------------- real-valued costs

def _same_f64(g, o):
    """Objectives and the cost are exact sums rounded once (reading R26):
    bit for bit on both sides."""
    assert g.adopt == o.adopt
    assert g.incumbent_objective == o.incumbent_objective
    assert g.proposal_objective == o.proposal_objective
    assert g.materialization_cost == o.materialization_cost
    np.testing.assert_array_equal(g.proposal, o.proposal)
    np.testing.assert_array_equal(g.target, o.target)


@pytest.mark.parametrize("seed", range(20))
def test_replan_f64_random(oracle_mod, seed):
    rng = np.random.default_rng(1700 + seed)
    m = int(rng.integers(1, 6))
    n = int(rng.integers(1, 260))
    inst = W.random_instance(n, m, rng, kmax=int(rng.choice([3, 40, n + 2])),
                             source_dependent=bool(seed % 3))
    lam, w, f = W.real_valued(inst, seed, jitter=0.5)
    inc = (rng.random((m, n)) < rng.choice([0.0, 0.1, 0.5, 1.0])).astype(np.uint8)
    horizon = float(rng.choice([0.0, 0.37, 7.0, 1e6]))
    eps = 1e-9 * (float(np.sum(lam * w)) + 1.0)
    kw = dict(epsilon=eps, n_starts=int(rng.integers(1, 4)),
              max_rounds=int(rng.integers(0, 3)),
              order_seed=int(rng.integers(0, 2 ** 62)))
    g = B.pp_replan_f64(inst.parent, lam, w, f, inst.cap, inc, horizon, **kw)
    o = oracle_mod.replan_f64(inst.parent, lam, w, f, inst.cap, inc, horizon, **kw)
    _same_f64(g, o)


def test_replan_f64_tree2k_routing_shift(oracle_mod):
    inst = W.make_workload("tree2k")
    lam, w, f = W.real_valued(inst, 4)
    eps = 1e-9 * float(np.sum(lam * w))
    kw = dict(epsilon=eps, n_starts=inst.n_starts, max_rounds=inst.max_rounds,
              order_seed=inst.order_seed)
    old = oracle_mod.plan_f64(inst.parent, lam, w, f, inst.cap, **kw)
    shifted = np.roll(lam, 1, axis=0)  # every request routed to the next worker
    for horizon in (0.5, 100.0, 1e6):
        g = B.pp_replan_f64(inst.parent, shifted, w, f, inst.cap, old.target,
                            horizon, **kw)
        o = oracle_mod.replan_f64(inst.parent, shifted, w, f, inst.cap, old.target,
                                  horizon, **kw)
        _same_f64(g, o)
