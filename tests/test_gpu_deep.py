"""GPU parity on deep trees whose pending skip rows exceed the DP sweep's
LDS slots (Eq. 9 has no depth bound; the paper's multi-turn workloads grow
long conversations that branch).  The sweep then spills the long-lived rows
to device memory and restores them (the schedule is replayed on the CPU in
test_sweep_layout.py); here the GPU must match the oracle bit for bit."""

import numpy as np
import pytest

from paper_2608_01655_amd import binding as B
from paper_2608_01655_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _say_case(request):
    print(f"\n[case] {request.node.name}", flush=True)
    yield


def _deep_trees():
    rng = np.random.default_rng(2024)
    trees = [("caterpillar300", W.caterpillar(300)),
             ("caterpillar1000", W.caterpillar(1000))]
    for q in range(3):
        trees.append((f"conversation{q}",
                      W.regenerated_conversation(int(rng.integers(1500, 5000)), rng)))
    return trees


TREES = _deep_trees()


def test_trees_spill():
    for name, parent in TREES:
        assert B.pp_sweep_spills(parent)[0] > 0, name


@pytest.mark.parametrize("idx", range(len(TREES)))
@pytest.mark.parametrize("cells", ["1", "2", "4"])
def test_rooted_dp_deep(oracle_mod, idx, cells, monkeypatch):
    monkeypatch.setenv("PP_DP_CELLS", cells)
    name, parent = TREES[idx]
    rng = np.random.default_rng(idx * 7 + int(cells))
    n = parent.shape[0]
    for k in (1, 63, 200, 700, n):
        for hi in (3, 10 ** 6):
            profit = rng.integers(0, hi, size=n).astype(np.int64)
            sel, val = B.pp_rooted_dp(parent, profit, k)
            osel, oval = oracle_mod.rooted_dp(parent, profit, k)
            assert val == oval, (name, k)
            np.testing.assert_array_equal(sel, osel)


@pytest.mark.parametrize("idx", range(len(TREES)))
@pytest.mark.parametrize("cells", [None, "2", "4"])
def test_plan_deep(oracle_mod, idx, cells, monkeypatch):
    if cells:
        monkeypatch.setenv("PP_DP_CELLS", cells)
    name, parent = TREES[idx]
    rng = np.random.default_rng(900 + idx)
    inst = W.random_instance(0, 3, rng, kmax=300, parent=parent,
                             source_dependent=bool(idx % 2))
    kw = dict(n_starts=2, max_rounds=0, order_seed=idx)
    g = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost, inst.fetch_cost,
                  inst.cap, **kw)
    o = oracle_mod.plan(inst.parent, inst.demand, inst.recompute_cost,
                        inst.fetch_cost, inst.cap, **kw)
    assert g.objective == o.objective
    assert g.start_sweeps.tolist() == o.start_sweeps.tolist()
    np.testing.assert_array_equal(g.target, o.target)


def test_plan_f64_deep(oracle_mod):
    name, parent = TREES[2]
    rng = np.random.default_rng(77)
    inst = W.random_instance(0, 3, rng, kmax=400, parent=parent)
    lam, w, f = W.real_valued(inst, 5, jitter=0.5)
    kw = dict(n_starts=2, max_rounds=0, order_seed=3, epsilon=0.0)
    g = B.pp_plan_f64(inst.parent, lam, w, f, inst.cap, **kw)
    o = oracle_mod.plan_f64(inst.parent, lam, w, f, inst.cap, **kw)
    assert g.objective == o.objective
    assert g.start_sweeps.tolist() == o.start_sweeps.tolist()
    np.testing.assert_array_equal(g.target, o.target)
