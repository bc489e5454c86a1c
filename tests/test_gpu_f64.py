"""GPU parity of the real-valued planner (Algorithm 1 on IEEE doubles with
the refinement tolerance epsilon) against the CPU oracle.

On integer-valued doubles every sum is exact, so the GPU must reproduce the
integer planner bit for bit -- checked on all five benchmark workloads at
full size against the oracle's stored plans.  On real values everything is
bit-exact too: profits, DP values, standalone scores, orders, sweep and
accept counts, placements, and the objectives, which both sides evaluate as
the exact sum of their rounded terms (reading R26), so that no decision
depends on a summation order -- also at epsilon = 0, where a replacement of
exactly equal value must be rejected.
"""

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


def _same_real(g, o):
    np.testing.assert_array_equal(g.standalone, o.standalone)
    np.testing.assert_array_equal(g.orders, o.orders)
    np.testing.assert_array_equal(g.start_sweeps, o.start_sweeps)
    np.testing.assert_array_equal(g.start_accepts, o.start_accepts)
    np.testing.assert_array_equal(g.start_objective, o.start_objective)
    assert g.best_start == o.best_start
    assert g.updates == o.updates and g.dp_cells == o.dp_cells
    assert g.objective == o.objective
    np.testing.assert_array_equal(g.target, o.target)


@pytest.mark.parametrize("seed", range(30))
def test_rooted_dp_f64_bit_exact(oracle_mod, seed):
    rng = np.random.default_rng(300 + seed)
    n = int(rng.integers(1, 3000))
    parent = W.random_forest(n, rng, p_root=float(rng.choice([0.0, 0.05, 0.3])))
    if seed % 3 == 0:
        profit = rng.integers(0, 5, size=n) / 64.0  # exact sums, many ties
    else:
        profit = rng.uniform(0.0, 1.0, size=n) * 10.0 ** rng.integers(-2, 7)
    k = int(rng.choice([1, 7, 64, 65, 300, n, n + 3]))
    sel, val = B.pp_rooted_dp_f64(parent, profit, k)
    osel, oval = oracle_mod.rooted_dp_f64(parent, profit, k)
    assert val == oval
    np.testing.assert_array_equal(sel, osel)


@pytest.mark.parametrize("seed", range(30))
def test_plan_f64_random_reals(oracle_mod, seed):
    rng = np.random.default_rng(800 + seed)
    m = int(rng.integers(1, 6))
    n = int(rng.integers(1, 260))
    inst = W.random_instance(n, m, rng, kmax=int(rng.choice([3, 40, n + 2])),
                             source_dependent=bool(seed % 4))
    lam, w, f = W.real_valued(inst, seed, jitter=0.5)
    kw = dict(n_starts=int(rng.integers(0, 4)), max_rounds=int(rng.integers(0, 3)),
              order_seed=int(rng.integers(0, 2 ** 62)),
              flags=B.PP_F_NO_REFINE if seed % 5 == 0 else 0)
    scale = float(np.sum(lam * w)) + 1.0
    eps = 1e-9 * scale
    g = B.pp_plan_f64(inst.parent, lam, w, f, inst.cap, epsilon=eps, **kw)
    o = oracle_mod.plan_f64(inst.parent, lam, w, f, inst.cap, epsilon=eps, **kw)
    _same_real(g, o)


def _valid_local_optimum(oracle_mod, parent, lam, w, f, cap, target):
    """Every row parent-closed and within capacity, and no worker's exact
    replacement (its marginals against the others, the rooted-tree DP)
    raises the exact objective: the placement refinement stops at."""
    from fractions import Fraction

    m, n = lam.shape
    for h in range(m):
        row = target[h]
        assert int(row.sum()) <= min(int(cap[h]), n)
        for v in np.flatnonzero(row):
            assert parent[v] < 0 or row[parent[v]], f"worker {h}: parent of {v} missing"

    def exact_g(t):
        best = np.zeros((m, n))
        for hh in range(m):
            for r in range(m):
                q = w[r] if hh == r else np.maximum(w[r] - f[hh, r], 0.0)
                best[r] = np.where(t[hh] != 0, np.maximum(best[r], q), best[r])
        return sum((Fraction(float(x)) for x in (lam * best).ravel()), Fraction(0))

    g = exact_g(target)
    for h in range(m):
        t = target.copy()
        t[h] = 0
        p = oracle_mod.marginal_f64(lam, w, f, t, h)
        t[h] = oracle_mod.rooted_dp_f64(parent, p, int(cap[h]))[0]
        assert exact_g(t) <= g


@pytest.mark.parametrize("seed", range(40))
def test_plan_f64_zero_tolerance_matches_oracle(oracle_mod, seed):
    """epsilon = 0 on real values (Algorithm 1's strict test with no slack):
    bit-exact against the oracle, including the replacements that differ
    from the worker's set only by chunks of zero marginal value -- exactly
    the same objective, to be rejected whatever two rounded sums would say
    -- and the result is a valid local optimum."""
    rng = np.random.default_rng(800 + seed)
    m = int(rng.integers(2, 6))
    n = int(rng.integers(5, 200))
    inst = W.random_instance(n, m, rng, kmax=int(rng.choice([3, 40, n + 2])),
                             source_dependent=bool(seed % 4))
    lam, w, f = W.real_valued(inst, seed, jitter=0.5)
    kw = dict(n_starts=int(rng.integers(1, 4)), max_rounds=0,
              order_seed=int(rng.integers(0, 2 ** 62)))
    g = B.pp_plan_f64(inst.parent, lam, w, f, inst.cap, epsilon=0.0, **kw)
    o = oracle_mod.plan_f64(inst.parent, lam, w, f, inst.cap, epsilon=0.0, **kw)
    _same_real(g, o)
    if seed % 4 == 0:
        _valid_local_optimum(oracle_mod, inst.parent, lam, w, f, inst.cap, g.target)


def _golden(name):
    with open(GOLDEN) as fh:
        return json.load(fh)[name]


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_integer_valued_workloads_match_integer_golden(name):
    """Every workload at full size, as doubles with epsilon = 0: the
    real-valued path must reproduce the integer oracle's stored plan."""
    inst = W.make_workload(name)
    gold = _golden(name)
    p = B.pp_plan_f64(inst.parent, inst.demand.astype(np.float64),
                      inst.recompute_cost.astype(np.float64),
                      inst.fetch_cost.astype(np.float64), inst.cap, epsilon=0.0,
                      n_starts=inst.n_starts, max_rounds=inst.max_rounds,
                      order_seed=inst.order_seed)
    assert p.objective == float(gold["objective"])
    assert p.best_start == gold["best_start"]
    assert p.standalone.tolist() == [float(x) for x in gold["standalone"]]
    assert p.orders.tolist() == gold["orders"]
    assert p.start_objective.tolist() == [float(x) for x in gold["start_objective"]]
    assert p.start_sweeps.tolist() == gold["start_sweeps"]
    assert p.start_accepts.tolist() == gold["start_accepts"]
    assert (p.updates, p.dp_cells) == (gold["updates"], gold["dp_cells"])
    rows = [hashlib.sha256(np.ascontiguousarray(p.target[h]).tobytes()).hexdigest()
            for h in range(inst.m)]
    assert rows == gold["target_row_sha256"]


def test_device_entry_rag10k_real_valued(oracle_mod):
    """The device-resident entry point on the 10,000-chunk RAG-shaped tree in
    milliseconds and requests, against the oracle."""
    import torch

    inst = W.make_workload("rag10k")
    lam, w, f = W.real_valued(inst, 1)
    eps = 1e-6 * float(np.sum(lam * w))
    dev = torch.device("cuda:0")
    tl = torch.from_numpy(lam).to(dev)
    tw = torch.from_numpy(w).to(dev)
    tf = torch.from_numpy(f).to(dev)
    tgt = torch.zeros((inst.m, inst.n), dtype=torch.uint8, device=dev)
    ctx = B.Context(0)
    kw = dict(n_starts=inst.n_starts, max_rounds=inst.max_rounds,
              order_seed=inst.order_seed)
    first = None
    for rep in range(2):  # a warm context must give the same answer
        g = ctx.pp_plan_f64_device(inst.parent, tl, tw, tf, inst.cap, tgt,
                                   epsilon=eps, flags=B.PP_F_TIME_KERNELS, **kw)
        g.target = tgt.cpu().numpy()
        if first is None:
            first = g
        else:
            assert g.objective == first.objective
            np.testing.assert_array_equal(g.target, first.target)
    ctx.close()
    o = oracle_mod.plan_f64(inst.parent, lam, w, f, inst.cap, epsilon=eps, **kw)
    _same_real(first, o)


def test_cells_per_lane_do_not_change_the_result(oracle_mod):
    """One, two or four DP cells per lane: the same real-valued plan, equal
    to the oracle's."""
    inst = W.make_workload("tree2k")
    lam, w, f = W.real_valued(inst, 2)
    eps = 1e-9 * float(np.sum(lam * w))
    kw = dict(n_starts=inst.n_starts, max_rounds=inst.max_rounds,
              order_seed=inst.order_seed)
    o = oracle_mod.plan_f64(inst.parent, lam, w, f, inst.cap, epsilon=eps, **kw)
    for cells in ("1", "2", "4"):
        os.environ["PP_DP_CELLS"] = cells
        try:
            g = B.pp_plan_f64(inst.parent, lam, w, f, inst.cap, epsilon=eps, **kw)
        finally:
            del os.environ["PP_DP_CELLS"]
        _same_real(g, o)


def test_tree50k_real_valued_golden():
    """The 50,000-chunk, 16-worker benchmark tree in the paper's units, at
    the benchmark's start settings, through the device entry point, against
    the oracle's stored real-valued plan."""
    import torch

    with open(os.path.join(os.path.dirname(GOLDEN), "plans_f64.json")) as fh:
        gold = json.load(fh)["tree50k"]
    inst = W.make_workload("tree50k")
    lam, w, f = W.real_valued(inst, 1)
    digest = hashlib.sha256(lam.tobytes() + w.tobytes() + f.tobytes()).hexdigest()
    assert digest == gold["inputs_sha256"]
    eps = float.fromhex(gold["epsilon"])
    dev = torch.device("cuda:0")
    tgt = torch.zeros((inst.m, inst.n), dtype=torch.uint8, device=dev)
    ctx = B.Context(0)
    p = ctx.pp_plan_f64_device(inst.parent, torch.from_numpy(lam).to(dev),
                               torch.from_numpy(w).to(dev),
                               torch.from_numpy(f).to(dev), inst.cap, tgt,
                               epsilon=eps, n_starts=inst.n_starts,
                               max_rounds=inst.max_rounds,
                               order_seed=inst.order_seed)
    target = tgt.cpu().numpy()
    ctx.close()
    assert p.standalone.tolist() == [float.fromhex(x) for x in gold["standalone"]]
    assert p.orders.tolist() == gold["orders"]
    assert p.start_sweeps.tolist() == gold["start_sweeps"]
    assert p.start_accepts.tolist() == gold["start_accepts"]
    assert p.best_start == gold["best_start"]
    assert (p.updates, p.dp_cells) == (gold["updates"], gold["dp_cells"])
    assert p.start_objective.tolist() == [float.fromhex(x) for x in gold["start_objective"]]
    assert p.objective == float.fromhex(gold["objective"])
    rows = [hashlib.sha256(np.ascontiguousarray(target[h]).tobytes()).hexdigest()
            for h in range(inst.m)]
    assert rows == gold["target_row_sha256"]


@pytest.mark.parametrize("seed", range(20))
def test_safeguards_f64_random(oracle_mod, seed):
    """Comparator safeguards on real requester-side costs (one fetch cost
    per requester and chunk, the same from every source)."""
    rng = np.random.default_rng(950 + seed)
    m = int(rng.integers(1, 6))
    n = int(rng.integers(1, 260))
    inst = W.random_instance(n, m, rng, kmax=int(rng.choice([3, 40, n + 2])),
                             source_dependent=False)
    lam, w, f = W.real_valued(inst, seed, jitter=0.5)
    # one factor per requester and chunk keeps the costs requester-side
    f = np.broadcast_to(f.max(axis=0)[None], f.shape).copy()
    for i in range(m):
        f[i, i] = 0.0
    if seed % 4 == 0 and m > 2:
        f[1, 2][f[1, 2] == 0.0] = -0.0  # equal as values to +0.0
    eps = 1e-9 * (float(np.sum(lam * w)) + 1.0)
    flags = B.PP_F_SAFEGUARDS | (B.PP_F_NO_REFINE if seed % 2 else 0)
    kw = dict(n_starts=int(rng.integers(1, 4)), max_rounds=int(rng.integers(0, 3)),
              flags=flags)
    g = B.pp_plan_f64(inst.parent, lam, w, f, inst.cap, epsilon=eps, **kw)
    o = oracle_mod.plan_f64(inst.parent, lam, w, f, inst.cap, epsilon=eps, **kw)
    assert o.safeguards_run and g.safeguards_run
    assert g.safeguard_objective == o.safeguard_objective
    _same_real(g, o)


def test_safeguards_f64_winning_candidates(oracle_mod):
    """Instances where a comparator beats a single greedy start."""
    found = 0
    for seed in range(3000):
        rng = np.random.default_rng(20000 + seed)
        m = int(rng.integers(2, 4))
        inst = W.random_instance(int(rng.integers(3, 12)), m, rng, kmax=5,
                                 source_dependent=False, value_range=20)
        lam, w, f = W.real_valued(inst, seed, jitter=0.3)
        f = np.broadcast_to(f.max(axis=0)[None], f.shape).copy()
        for i in range(m):
            f[i, i] = 0.0
        kw = dict(n_starts=1, flags=B.PP_F_SAFEGUARDS | B.PP_F_NO_REFINE,
                  epsilon=1e-9)
        o = oracle_mod.plan_f64(inst.parent, lam, w, f, inst.cap, **kw)
        if o.best_start < 1:
            continue
        g = B.pp_plan_f64(inst.parent, lam, w, f, inst.cap, **kw)
        _same_real(g, o)
        found += 1
        if found == 6:
            break
    assert found > 0


@pytest.mark.parametrize("m", [4, 8])
def test_paper_runtime_configuration_matches_oracle(oracle_mod, m):
    """The paper's solver-runtime configuration at n = 10,000 (k = 128, the
    paper's default start set: all 24 orders at M = 4, 8 starts at M = 8;
    the bench checks M = 16 the same way),
    real-valued, refinement to convergence: the plan the bench times is the
    oracle's, bit for bit."""
    inst = W.runtime_instance(m)
    lam, w, f = W.real_valued(inst, 1)
    eps = 1e-9 * float(np.sum(lam * w))
    kw = dict(epsilon=eps, n_starts=inst.n_starts, max_rounds=inst.max_rounds,
              order_seed=inst.order_seed)
    g = B.pp_plan_f64(inst.parent, lam, w, f, inst.cap, **kw)
    o = oracle_mod.plan_f64(inst.parent, lam, w, f, inst.cap, **kw)
    _same_real(g, o)
    assert g.n_starts == (24 if m == 4 else 8)


@pytest.mark.parametrize("chains,rounds", [(3, 2), (5, 0)])
def test_f64_speculation_into_the_next_sweep(oracle_mod, monkeypatch, chains, rounds):
    """Real-valued refinement with a few updates per launch, so that
    speculation reaches into starts' next sweeps at several points, with
    and without a sweep cap: the oracle's plan, bit for bit."""
    inst = W.runtime_instance(4)
    lam, w, f = W.real_valued(inst, 2)
    eps = 1e-9 * float(np.sum(lam * w))
    kw = dict(epsilon=eps, n_starts=6, max_rounds=rounds, order_seed=inst.order_seed)
    monkeypatch.setenv("PP_SPEC_CHAINS", str(chains))
    g = B.pp_plan_f64(inst.parent, lam, w, f, inst.cap, **kw)
    o = oracle_mod.plan_f64(inst.parent, lam, w, f, inst.cap, **kw)
    _same_real(g, o)


@pytest.mark.parametrize("seed", range(15))
def test_plan_f64_random_launch_budgets(oracle_mod, monkeypatch, seed):
    """Real-valued random plans with 2 to 64 updates per refinement launch:
    the oracle's plan, bit for bit."""
    rng = np.random.default_rng(6100 + seed)
    m = int(rng.integers(1, 7))
    n = int(rng.integers(1, 300))
    inst = W.random_instance(n, m, rng, kmax=int(rng.choice([3, 40, n + 2])),
                             source_dependent=bool(seed % 3))
    lam, w, f = W.real_valued(inst, seed, jitter=0.5)
    kw = dict(n_starts=int(rng.integers(0, 6)), max_rounds=int(rng.integers(0, 4)),
              order_seed=int(rng.integers(0, 2 ** 62)))
    eps = 1e-9 * (float(np.sum(lam * w)) + 1.0)
    monkeypatch.setenv("PP_SPEC_CHAINS", str(int(rng.choice([2, 3, 5, 64]))))
    g = B.pp_plan_f64(inst.parent, lam, w, f, inst.cap, epsilon=eps, **kw)
    o = oracle_mod.plan_f64(inst.parent, lam, w, f, inst.cap, epsilon=eps, **kw)
    _same_real(g, o)


def test_f64_device_entry_input_errors_then_a_valid_plan(oracle_mod):
    """Real-valued device entry: a negative, NaN or infinite value in any of
    the three inputs (late blocks of the check) is PP_E_RANGE, a cyclic
    parent array PP_E_TREE; the same context then plans valid inputs as the
    oracle does."""
    import torch

    rng = np.random.default_rng(32)
    inst = W.random_instance(3000, 4, rng, kmax=200, shuffle=False)
    lam, w, f = W.real_valued(inst, 4, jitter=0.5)
    dev = torch.device("cuda:0")
    ctx = B.Context(0)
    tgt = torch.zeros((inst.m, inst.n), dtype=torch.uint8, device=dev)
    eps = 1e-9 * (float(np.sum(lam * w)) + 1.0)

    def run(a, b, c, parent=inst.parent):
        t = [torch.from_numpy(np.ascontiguousarray(x)).to(dev) for x in (a, b, c)]
        return ctx.pp_plan_f64_device(parent, *t, inst.cap, tgt, epsilon=eps, n_starts=2,
                                      order_seed=5)

    for which, idx, val in ((0, (3, 2999), -1.0), (1, (2, 1777), float("nan")),
                            (2, (3, 2, 2998), float("inf"))):
        arrs = [lam.copy(), w.copy(), f.copy()]
        arrs[which][idx] = val
        with pytest.raises(B.PPError) as e:
            run(*arrs)
        assert e.value.code == B.PP_E_RANGE
    cyc = inst.parent.copy(); cyc[0] = 5; cyc[5] = 0
    with pytest.raises(B.PPError) as e:
        run(lam, w, f, parent=cyc)
    assert e.value.code == B.PP_E_TREE
    import dataclasses

    g = run(lam, w, f)
    g = dataclasses.replace(g, target=tgt.cpu().numpy())
    o = oracle_mod.plan_f64(inst.parent, lam, w, f, inst.cap, epsilon=eps, n_starts=2,
                            order_seed=5)
    _same_real(g, o)
    ctx.close()
