"""GPU parity of the whole planner (Algorithm 1) against the CPU oracle:
identical placements, objective, per-start objectives, sweep and accept
counts, standalone scores, orders and work counters -- bit-exact."""

import hashlib
import json
import os

import numpy as np
import pytest

from paper_2608_01655_amd import binding as B
from paper_2608_01655_amd import workloads as W

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "plans.json")


@pytest.fixture(autouse=True)
def _say_case(request):
    print(f"\n[case] {request.node.name}", flush=True)
    yield


def _same(gpu, ora):
    assert gpu.objective == ora.objective
    np.testing.assert_array_equal(gpu.standalone, ora.standalone)
    np.testing.assert_array_equal(gpu.orders, ora.orders)
    np.testing.assert_array_equal(gpu.start_objective, ora.start_objective)
    np.testing.assert_array_equal(gpu.start_sweeps, ora.start_sweeps)
    np.testing.assert_array_equal(gpu.start_accepts, ora.start_accepts)
    assert gpu.best_start == ora.best_start
    assert gpu.updates == ora.updates
    assert gpu.dp_cells == ora.dp_cells
    np.testing.assert_array_equal(gpu.target, ora.target)


def _plan_both(oracle_mod, inst, **kw):
    args = dict(n_starts=inst.n_starts, max_rounds=inst.max_rounds,
                order_seed=inst.order_seed)
    args.update(kw)
    g = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost,
                  inst.fetch_cost, inst.cap, **args)
    orders = args.pop("orders", None)
    o = oracle_mod.plan_instance(inst, orders_in=orders, threads=8, **args)
    return g, o


@pytest.mark.parametrize("seed", range(40))
def test_plan_random(oracle_mod, seed):
    rng = np.random.default_rng(seed)
    m = int(rng.integers(1, 7))
    n = int(rng.integers(1, 300))
    inst = W.random_instance(n, m, rng, kmax=int(rng.choice([3, 40, 200, n + 2])),
                             source_dependent=bool(seed % 4),
                             value_range=int(rng.choice([5, 100, 10 ** 5])))
    g, o = _plan_both(oracle_mod, inst, n_starts=int(rng.integers(0, 5)),
                      max_rounds=int(rng.integers(0, 4)),
                      order_seed=int(rng.integers(0, 2 ** 62)))
    _same(g, o)


@pytest.mark.parametrize("seed", range(30))
def test_plan_random_launch_budgets(oracle_mod, monkeypatch, seed):
    """Random small plans with 2 to 64 updates per refinement launch (so
    that speculation, within a sweep and into the next, stops at every
    kind of boundary: launch budget, sweep cap, workers without capacity,
    a single worker) and a few stage blocks per launch: the oracle's plan."""
    rng = np.random.default_rng(5000 + seed)
    m = int(rng.integers(1, 9))
    n = int(rng.integers(1, 400))
    inst = W.random_instance(n, m, rng, kmax=int(rng.choice([3, 40, 200, n + 2])),
                             source_dependent=bool(seed % 3),
                             value_range=int(rng.choice([5, 100, 10 ** 5])))
    monkeypatch.setenv("PP_SPEC_CHAINS", str(int(rng.choice([2, 3, 5, 9, 64]))))
    monkeypatch.setenv("PP_SPEC_BLOCKS", str(int(rng.choice([1, 3, 8, 512]))))
    g, o = _plan_both(oracle_mod, inst, n_starts=int(rng.integers(0, 7)),
                      max_rounds=int(rng.integers(0, 4)),
                      order_seed=int(rng.integers(0, 2 ** 62)))
    _same(g, o)


def test_plan_flags_and_explicit_orders(oracle_mod):
    rng = np.random.default_rng(11)
    inst = W.random_instance(150, 4, rng, kmax=60)
    g, o = _plan_both(oracle_mod, inst, n_starts=3, flags=B.PP_F_NO_REFINE)
    _same(g, o)
    orders = np.array([[3, 2, 1, 0], [1, 3, 0, 2]], np.int32)
    g, o = _plan_both(oracle_mod, inst, n_starts=2, orders=orders)
    _same(g, o)


@pytest.mark.parametrize("name", ["tiny", "tree2k", "rag10k"])
def test_plan_small_workloads_live(oracle_mod, name):
    inst = W.make_workload(name)
    g, o = _plan_both(oracle_mod, inst)
    _same(g, o)


def _golden(name):
    with open(GOLDEN) as fh:
        return json.load(fh)[name]


def _check_golden(inst, gold, plan, target):
    assert inst.checksum() == gold["input_sha256"]
    assert plan.objective == gold["objective"]
    assert plan.best_start == gold["best_start"]
    assert plan.standalone.tolist() == gold["standalone"]
    assert plan.orders.tolist() == gold["orders"]
    assert plan.start_objective.tolist() == gold["start_objective"]
    assert plan.start_sweeps.tolist() == gold["start_sweeps"]
    assert plan.start_accepts.tolist() == gold["start_accepts"]
    assert plan.updates == gold["updates"]
    assert plan.dp_cells == gold["dp_cells"]
    rows = [hashlib.sha256(np.ascontiguousarray(target[h]).tobytes()).hexdigest()
            for h in range(inst.m)]
    assert rows == gold["target_row_sha256"]


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_plan_workloads_golden(name):
    """All five workloads at full size against the oracle's stored plans."""
    inst = W.make_workload(name)
    gold = _golden(name)
    p = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost,
                  inst.fetch_cost, inst.cap, n_starts=inst.n_starts,
                  max_rounds=inst.max_rounds, order_seed=inst.order_seed)
    _check_golden(inst, gold, p, p.target)


@pytest.mark.parametrize("name", ["rag10k", "tree50k"])
def test_plan_device_path_golden(name):
    """The device-resident entry point (the one the bench times) on torch
    tensors, with kernel timing on."""
    import torch

    inst = W.make_workload(name)
    gold = _golden(name)
    dev = torch.device("cuda:0")
    lam = torch.from_numpy(inst.demand).to(dev)
    w = torch.from_numpy(inst.recompute_cost).to(dev)
    f = torch.from_numpy(inst.fetch_cost).to(dev)
    tgt = torch.zeros((inst.m, inst.n), dtype=torch.uint8, device=dev)
    ctx = B.Context(0)
    for rep in range(2):  # a warm context must give the same answer
        p = ctx.pp_plan_device(inst.parent, lam, w, f, inst.cap, tgt,
                               n_starts=inst.n_starts,
                               max_rounds=inst.max_rounds,
                               order_seed=inst.order_seed,
                               flags=B.PP_F_TIME_KERNELS)
        _check_golden(inst, gold, p, tgt.cpu().numpy())
        assert p.dp_launches > 0 and p.dp_kernel_ms > 0
    ctx.close()


def test_context_on_alternating_streams():
    """One context used on two streams in turn, for trees of different
    sizes (the staged tree-table uploads switch streams, wrap and grow):
    every plan is the stored one."""
    import torch

    dev = torch.device("cuda:0")
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    cases = []
    for name in ("tree2k", "tiny", "rag10k"):
        inst = W.make_workload(name)
        t = [torch.from_numpy(a).to(dev) for a in (inst.demand, inst.recompute_cost,
                                                   inst.fetch_cost)]
        cases.append((inst, _golden(name), t))
    torch.cuda.synchronize()
    ctx = B.Context(0)
    # (workload, stream): switches, and three rag10k plans in a row on one
    # stream (more than the staging buffer's first size)
    for ci, si in ((0, 0), (1, 1), (2, 0), (2, 0), (2, 0), (0, 1), (1, 1)):
        inst, gold, (lam, w, f) = cases[ci]
        st = streams[si]
        with torch.cuda.stream(st):
            tgt = torch.zeros((inst.m, inst.n), dtype=torch.uint8, device=dev)
            p = ctx.pp_plan_device(inst.parent, lam, w, f, inst.cap, tgt,
                                   n_starts=inst.n_starts, max_rounds=inst.max_rounds,
                                   order_seed=inst.order_seed, stream=st)
        st.synchronize()
        _check_golden(inst, gold, p, tgt.cpu().numpy())
    ctx.close()


def test_plan_is_deterministic():
    inst = W.make_workload("tree2k")
    a = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost, inst.fetch_cost,
                  inst.cap, n_starts=4, order_seed=2)
    for cells in ("1", "4"):
        os.environ["PP_DP_CELLS"] = cells
        try:
            b = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost,
                          inst.fetch_cost, inst.cap, n_starts=4, order_seed=2)
        finally:
            del os.environ["PP_DP_CELLS"]
        assert a.objective == b.objective
        np.testing.assert_array_equal(a.target, b.target)
        np.testing.assert_array_equal(a.start_objective, b.start_objective)


def test_stall_guard_reports_device_error(monkeypatch):
    """A tiny spin limit on the sweep's bounded stage-to-stage wait, forced
    from the host: the call either completes correctly or reports
    PP_E_DEVICE -- every kernel still exits normally."""
    inst = W.make_workload("tree2k")
    ref = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost,
                    inst.fetch_cost, inst.cap, n_starts=2)
    monkeypatch.setenv("PP_SPIN_LIMIT", "0")
    try:
        p = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost,
                      inst.fetch_cost, inst.cap, n_starts=2)
        assert p.objective == ref.objective
    except B.PPError as e:
        assert e.code == B.PP_E_DEVICE
    monkeypatch.delenv("PP_SPIN_LIMIT")
    p = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost,
                  inst.fetch_cost, inst.cap, n_starts=2)
    assert p.objective == ref.objective


def test_plan_maximum_workers(oracle_mod):
    """255 workers (the maximum): the standalone pass and every update span
    several launches of at most 64 chains."""
    rng = np.random.default_rng(255)
    inst = W.random_instance(30, 255, rng, kmax=6, value_range=50)
    g, o = _plan_both(oracle_mod, inst, n_starts=2, max_rounds=1)
    _same(g, o)


def test_plan_deep_caterpillar(oracle_mod):
    """A 250-level spine with a side leaf per level, each pending while the
    spine below it is swept (250 LDS slots)."""
    depth = 250
    parent = np.array([-1] + list(range(0, depth - 1)) + list(range(0, depth)),
                      np.int32)
    n = parent.shape[0]
    rng = np.random.default_rng(9)
    m = 3
    lam = rng.integers(0, 20, size=(m, n)).astype(np.int64)
    w = rng.integers(0, 20, size=(m, n)).astype(np.int64)
    f = rng.integers(0, 20, size=(m, m, n)).astype(np.int64)
    cap = np.array([40, 120, n], np.int32)
    g = B.pp_plan(parent, lam, w, f, cap, n_starts=2, max_rounds=0)
    o = oracle_mod.plan(parent, lam, w, f, cap, n_starts=2, max_rounds=0)
    _same(g, o)


def test_unchanged_workers_skip_their_sweep(oracle_mod, monkeypatch):
    """Refinement updates of workers whose inputs have not changed are
    resolved without a sweep: fewer cells swept, identical plan (without
    speculative sweeps, whose discarded updates add swept cells).  Without
    refinement every update but the first greedy one of each start is swept:
    that one (all sets still empty) adopts the standalone solve of the
    start's first worker."""
    monkeypatch.setenv("PP_NO_SPEC", "1")
    inst = W.make_workload("tree2k")
    g, o = _plan_both(oracle_mod, inst)
    _same(g, o)
    assert g.dp_cells_executed < g.dp_cells
    nr = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost, inst.fetch_cost,
                   inst.cap, n_starts=inst.n_starts, order_seed=inst.order_seed,
                   flags=B.PP_F_NO_REFINE)
    n = inst.n
    first = sum(n * min(int(inst.cap[order[0]]), n) for order in nr.orders)
    assert nr.dp_cells_executed == nr.dp_cells - first


@pytest.mark.parametrize("name,starts", [("tree2k", 1), ("tree2k", 2), ("rag10k", 3),
                                         ("tiny", 1), ("tree2k", 5)])
def test_speculative_sweeps(oracle_mod, monkeypatch, name, starts):
    """Refinement runs each start at its own position, passes over updates
    resolved without a sweep on the host, and fills each launch with
    speculative updates of later positions (the first accepted one is
    adopted, the rest computed again).  Same plan and statistics as without
    speculation and as the oracle; fewer DP launches."""
    inst = W.make_workload(name)
    args = dict(n_starts=starts, max_rounds=0, order_seed=inst.order_seed)
    g = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost, inst.fetch_cost,
                  inst.cap, flags=B.PP_F_TIME_KERNELS, **args)
    monkeypatch.setenv("PP_NO_SPEC", "1")
    q = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost, inst.fetch_cost,
                  inst.cap, flags=B.PP_F_TIME_KERNELS, **args)
    o = oracle_mod.plan_instance(inst, threads=8, **args)
    _same(g, o)
    _same(q, o)
    assert g.updates == q.updates and g.dp_cells == q.dp_cells
    if starts <= 4 and name != "tiny":
        assert g.dp_launches < q.dp_launches


@pytest.mark.parametrize("chains,rounds", [(2, 0), (3, 2), (6, 3), (6, 0), (64, 2), (64, 0)])
def test_speculation_into_the_next_sweep(oracle_mod, monkeypatch, chains, rounds):
    """A start whose sweep has accepted an update and whose remaining
    positions all fit the launch speculates positions of its next sweep
    (those whose workers are stale) unless the sweep cap ends it there:
    with a few or many updates per launch and with and without a cap, the
    plan and its statistics are the oracle's."""
    inst = W.make_workload("tree2k")
    args = dict(n_starts=2, max_rounds=rounds, order_seed=inst.order_seed)
    monkeypatch.setenv("PP_SPEC_CHAINS", str(chains))
    g = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost, inst.fetch_cost,
                  inst.cap, **args)
    o = oracle_mod.plan_instance(inst, threads=8, **args)
    _same(g, o)
    if rounds == 0:
        assert max(g.start_sweeps) >= 2


def test_stalled_sweep_is_run_again(oracle_mod, monkeypatch):
    """A DP sweep whose stage gives up its bounded wait for the neighbouring
    stage (forced from the host with a one-poll spin limit, so every kernel
    still exits normally) makes the library run the plan again with fewer
    stage blocks per launch and the default wait: the same plan as the
    oracle, with the restart reported."""
    inst = W.make_workload("tree2k")
    monkeypatch.setenv("PP_SPIN_LIMIT", "1")
    p = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost, inst.fetch_cost,
                  inst.cap, n_starts=inst.n_starts, max_rounds=inst.max_rounds,
                  order_seed=inst.order_seed)
    assert p.dp_restarts >= 1
    o = oracle_mod.plan_instance(inst)
    assert p.objective == o.objective
    np.testing.assert_array_equal(p.target, o.target)
    rng = np.random.default_rng(5)
    parent = W.random_forest(3000, rng)
    profit = rng.integers(0, 1000, size=3000).astype(np.int64)
    sel, val = B.pp_rooted_dp(parent, profit, 900)
    osel, oval = oracle_mod.rooted_dp(parent, profit, 900)
    assert val == oval
    np.testing.assert_array_equal(sel, osel)


def test_device_entry_input_errors_then_a_valid_plan(oracle_mod):
    """The device entry's input checks run on the GPU while the host builds
    the tree tables: a negative demand, recompute or fetch cost anywhere
    (here in late blocks of the check) is PP_E_RANGE, a sum of demand *
    recompute cost above INT64_MAX is PP_E_OVERFLOW, a cyclic parent array
    is PP_E_TREE even when values are bad too; the same context then plans
    valid inputs exactly as the oracle does."""
    import torch

    rng = np.random.default_rng(31)
    inst = W.random_instance(3000, 4, rng, kmax=200, shuffle=False)
    dev = torch.device("cuda:0")
    ctx = B.Context(0)
    tgt = torch.zeros((inst.m, inst.n), dtype=torch.uint8, device=dev)

    def run(lam, w, f, parent=inst.parent):
        t = [torch.from_numpy(np.ascontiguousarray(a)).to(dev) for a in (lam, w, f)]
        return ctx.pp_plan_device(parent, *t, inst.cap, tgt, n_starts=2, order_seed=5)

    cases = []
    lam = inst.demand.copy(); lam[3, 2999] = -1; cases.append(((lam, inst.recompute_cost, inst.fetch_cost), B.PP_E_RANGE))
    w = inst.recompute_cost.copy(); w[2, 1777] = -5; cases.append(((inst.demand, w, inst.fetch_cost), B.PP_E_RANGE))
    f = inst.fetch_cost.copy(); f[3, 2, 2998] = -1; cases.append(((inst.demand, inst.recompute_cost, f), B.PP_E_RANGE))
    big = inst.demand.copy(); big[0, :] = 2 ** 40
    wb = inst.recompute_cost.copy(); wb[0, :] = 2 ** 40
    cases.append(((big, wb, inst.fetch_cost), B.PP_E_OVERFLOW))
    for args, code in cases:
        with pytest.raises(B.PPError) as e:
            run(*args)
        assert e.value.code == code
    cyc = inst.parent.copy(); cyc[0] = 5; cyc[5] = 0
    with pytest.raises(B.PPError) as e:
        run(cases[0][0][0], inst.recompute_cost, inst.fetch_cost, parent=cyc)
    assert e.value.code == B.PP_E_TREE
    g = run(inst.demand, inst.recompute_cost, inst.fetch_cost)
    o = oracle_mod.plan(inst.parent, inst.demand, inst.recompute_cost, inst.fetch_cost,
                        inst.cap, n_starts=2, order_seed=5)
    assert g.objective == o.objective
    np.testing.assert_array_equal(tgt.cpu().numpy(), o.target)
    ctx.close()
