"""GPU parity of the comparator safeguards (Sec. IV-C, Algorithm 1:
Independent, Popularity and LocalDedup candidates for requester-side costs)
against the CPU oracle: placement, objective, returned candidate, candidate
objectives and work counters -- bit-exact."""

import numpy as np
import pytest

from paper_2608_01655_amd import binding as B
from paper_2608_01655_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _say_case(request):
    print(f"\n[case] {request.node.name}", flush=True)
    yield


def _same(g, o):
    assert g.objective == o.objective
    assert g.best_start == o.best_start
    assert g.updates == o.updates and g.dp_cells == o.dp_cells
    assert g.safeguards_run == o.safeguards_run
    assert tuple(g.safeguard_objective) == tuple(o.safeguard_objective)
    np.testing.assert_array_equal(g.start_objective, o.start_objective)
    np.testing.assert_array_equal(g.target, o.target)


def _both(oracle_mod, inst, n_starts, max_rounds, flags):
    g = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost, inst.fetch_cost,
                  inst.cap, n_starts=n_starts, max_rounds=max_rounds,
                  order_seed=inst.order_seed, flags=flags)
    o = oracle_mod.plan(inst.parent, inst.demand, inst.recompute_cost,
                        inst.fetch_cost, inst.cap, n_starts=n_starts,
                        max_rounds=max_rounds, order_seed=inst.order_seed,
                        flags=flags, threads=8)
    return g, o


@pytest.mark.parametrize("seed", range(30))
def test_safeguards_random(oracle_mod, seed):
    rng = np.random.default_rng(500 + seed)
    m = int(rng.integers(1, 6))
    n = int(rng.integers(1, 260))
    inst = W.random_instance(n, m, rng, kmax=int(rng.choice([3, 40, n + 2])),
                             source_dependent=False,
                             value_range=int(rng.choice([5, 100, 10 ** 5])))
    flags = B.PP_F_SAFEGUARDS | (B.PP_F_NO_REFINE if seed % 2 else 0)
    g, o = _both(oracle_mod, inst, int(rng.integers(1, 4)), int(rng.integers(0, 3)),
                 flags)
    assert o.safeguards_run
    _same(g, o)


def _winning_instances(oracle_mod, count):
    """Tiny requester-side instances where a comparator beats a single
    greedy start (found with the oracle)."""
    found = []
    for seed in range(2000):
        rng = np.random.default_rng(9000 + seed)
        m = int(rng.integers(2, 4))
        inst = W.random_instance(int(rng.integers(3, 12)), m, rng, kmax=5,
                                 source_dependent=False, value_range=20)
        o = oracle_mod.plan(inst.parent, inst.demand, inst.recompute_cost,
                            inst.fetch_cost, inst.cap, n_starts=1,
                            flags=B.PP_F_NO_REFINE | B.PP_F_SAFEGUARDS)
        if o.best_start >= 1:
            found.append(inst)
            if len(found) == count:
                break
    return found


def test_safeguard_wins_match(oracle_mod):
    cases = _winning_instances(oracle_mod, 8)
    assert cases, "no instance where a comparator wins"
    for inst in cases:
        g, o = _both(oracle_mod, inst, 1, 0, B.PP_F_NO_REFINE | B.PP_F_SAFEGUARDS)
        assert o.best_start >= 1
        _same(g, o)


def test_safeguards_tiny_workload(oracle_mod):
    inst = W.make_workload("tiny")
    g, o = _both(oracle_mod, inst, inst.n_starts, inst.max_rounds,
                 B.PP_F_SAFEGUARDS)
    assert o.safeguards_run
    _same(g, o)


def test_safeguards_single_worker(oracle_mod):
    rng = np.random.default_rng(77)
    inst = W.random_instance(120, 1, rng, kmax=30, source_dependent=False)
    g, o = _both(oracle_mod, inst, 1, 0, B.PP_F_SAFEGUARDS)
    assert o.safeguards_run
    _same(g, o)


def test_safeguards_noop_for_source_dependent(oracle_mod):
    rng = np.random.default_rng(5)
    inst = W.random_instance(200, 4, rng, kmax=40, source_dependent=True)
    g, o = _both(oracle_mod, inst, 2, 1, B.PP_F_SAFEGUARDS)
    assert not g.safeguards_run and not o.safeguards_run
    plain = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost,
                      inst.fetch_cost, inst.cap, n_starts=2, max_rounds=1)
    assert g.objective == plain.objective
    np.testing.assert_array_equal(g.target, plain.target)
    _same(g, o)


def test_safeguards_device_entry_rag(oracle_mod):
    """The device entry point on the 10,000-chunk RAG-shaped tree with a
    requester-side fetch cost (every source the same), 8 workers."""
    import torch

    inst = W.make_workload("rag10k")
    m, n = inst.demand.shape
    f = W.requester_fetch(m, n, 60_000)
    dev = torch.device("cuda:0")
    lam = torch.from_numpy(inst.demand).to(dev)
    w = torch.from_numpy(inst.recompute_cost).to(dev)
    ft = torch.from_numpy(f).to(dev)
    tgt = torch.zeros((m, n), dtype=torch.uint8, device=dev)
    ctx = B.Context(0)
    g = ctx.pp_plan_device(inst.parent, lam, w, ft, inst.cap, tgt, n_starts=2,
                           max_rounds=1, order_seed=inst.order_seed,
                           flags=B.PP_F_SAFEGUARDS)
    o = oracle_mod.plan(inst.parent, inst.demand, inst.recompute_cost, f,
                        inst.cap, n_starts=2, max_rounds=1,
                        order_seed=inst.order_seed, flags=B.PP_F_SAFEGUARDS,
                        threads=8)
    assert o.safeguards_run and g.safeguards_run
    assert g.objective == o.objective and g.best_start == o.best_start
    assert tuple(g.safeguard_objective) == tuple(o.safeguard_objective)
    np.testing.assert_array_equal(tgt.cpu().numpy(), o.target)
