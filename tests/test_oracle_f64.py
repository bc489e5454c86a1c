"""Oracle pins of the real-valued planner (Algorithm 1 with its floating-point
tolerance epsilon; reading R24).  CPU only.

Pinned against what the mathematics fixes, independently of the oracle's
code: on integer-valued doubles every sum is exact, so the planner must
reproduce the integer oracle (itself pinned by exhaustive search and the
paper's theorems) bit for bit; on dyadic profits the DP must return the
exhaustive optimum and its tie rule (R1); on generic reals the DP must reach
the exhaustive optimum within rounding, the objective must match Eq. 6
evaluated with NumPy, Proposition 1's exact-gain identity must hold within
rounding, every fixed-order greedy start must reach half the exhaustive joint
optimum (Theorem 3), and the tolerance must gate refinement as stated.

Reading R26 (G is the exact sum of its rounded terms) is pinned by Python's
math.fsum, which returns the correctly rounded exact sum of its inputs, by
rounding edge cases (ties to even, denormals, overflow), and by an
independent driver of Algorithm 1 that evaluates G with exact rationals
(fractions.Fraction) and must make every acceptance decision the oracle
makes, including the cases where two rounded sums would disagree.
"""

import itertools
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2608_01655_amd import workloads as W
from tests import bruteforce as bf


def as_f64(inst):
    return (inst.demand.astype(np.float64), inst.recompute_cost.astype(np.float64),
            inst.fetch_cost.astype(np.float64))


def real_instance(seed, n_max=60, m_max=4, source_dependent=True):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, n_max + 1))
    m = int(rng.integers(1, m_max + 1))
    parent = W.random_forest(n, rng)
    lam = rng.gamma(0.7, 3.0, size=(m, n))
    lam[rng.random((m, n)) < 0.2] = 0.0
    w = rng.uniform(0.0, 50.0, size=(m, n))
    if source_dependent:
        f = rng.uniform(0.0, 60.0, size=(m, m, n))
    else:
        fr = rng.uniform(0.0, 60.0, size=(m, n))
        f = np.broadcast_to(fr[None], (m, m, n)).copy()
    for i in range(m):
        f[i, i] = 0.0
    cap = rng.integers(0, n + 2, size=m).astype(np.int32)
    return parent, lam, w, f, cap


# -------------------------------------------------------------- RootedDP

@pytest.mark.parametrize("seed", range(60))
def test_dp_dyadic_profits_match_exhaustive_and_tie_rule(seed):
    """Profits k/1024 make every sum exact: the set and value must be the
    exhaustive optimum with R1's lexicographic tie rule."""
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 11))
    parent = W.random_forest(n, rng)
    units = rng.integers(0, 4, size=n)  # many ties
    profit = units / 1024.0
    k = int(rng.integers(0, n + 2))
    sel, val = oracle.rooted_dp_f64(parent, profit, k)
    want_sel, want_units = bf.best_closed_set(parent, [int(u) for u in units], k)
    assert val == want_units / 1024.0
    np.testing.assert_array_equal(sel, want_sel)


@pytest.mark.parametrize("seed", range(60))
def test_dp_generic_reals_reach_the_exhaustive_optimum(seed):
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(1, 11))
    parent = W.random_forest(n, rng)
    profit = rng.uniform(0.0, 1.0, size=n) * 10.0 ** rng.integers(-3, 6)
    k = int(rng.integers(0, n + 2))
    sel, val = oracle.rooted_dp_f64(parent, profit, k)
    sums = [(math.fsum(profit[s]), tuple(s)) for s in bf.closed_sets(parent, k)]
    best = max(v for v, _ in sums)
    assert val == pytest.approx(best, rel=1e-12, abs=0.0)
    # generic reals: the optimum is unique and the DP returns it
    winners = [s for v, s in sums if v == best]
    assert len(winners) == 1
    np.testing.assert_array_equal(sel.astype(bool), np.array(winners[0]))
    # the returned set is closed and within the budget
    assert sel.sum() <= k
    for v in range(n):
        if sel[v] and parent[v] >= 0:
            assert sel[parent[v]]


# ---------------------------------------------------- objective, marginal

def objective_numpy(lam, w, f, tgt):
    """Eq. 6 with NumPy: q per Eq. 5, best holder per (requester, chunk)."""
    m, n = lam.shape
    q = np.empty((m, m, n))
    for h in range(m):
        for r in range(m):
            q[h, r] = w[r] if h == r else np.maximum(w[r] - f[h, r], 0.0)
    best = np.max(np.where(tgt.astype(bool)[:, None, :], q, 0.0), axis=0)
    return float(np.sum(lam * best))


@pytest.mark.parametrize("seed", range(30))
def test_objective_matches_eq6(seed):
    parent, lam, w, f, cap = real_instance(seed)
    rng = np.random.default_rng(seed)
    tgt = (rng.random(lam.shape) < 0.4).astype(np.uint8)
    got = oracle.objective_f64(lam, w, f, tgt)
    assert got == pytest.approx(objective_numpy(lam, w, f, tgt), rel=1e-12)


def eq6_terms(lam, w, f, tgt):
    """The rounded terms lam_m(b) * max over holders h of q_{m<-h}(b) (Eq. 5,
    Eq. 6; 0 where nobody holds b), as NumPy computes them."""
    m, n = lam.shape
    best = np.zeros((m, n))
    for h in range(m):
        for r in range(m):
            q = w[r] if h == r else np.maximum(w[r] - f[h, r], 0.0)
            best[r] = np.where(tgt[h] != 0, np.maximum(best[r], q), best[r])
    return (lam * best).ravel()


@pytest.mark.parametrize("seed", range(40))
def test_objective_is_the_correctly_rounded_exact_sum(seed):
    """R26: G is the exact sum of the rounded terms, rounded once: it equals
    math.fsum of the same terms bit for bit, at every magnitude."""
    parent, lam, w, f, cap = real_instance(9000 + seed, n_max=200, m_max=5)
    rng = np.random.default_rng(seed)
    if seed % 4 == 1:  # terms spread over many binades
        lam = lam * np.exp2(rng.integers(-60, 60, size=lam.shape))
    if seed % 4 == 2:  # denormal and tiny terms only
        lam = lam * 2.0 ** -1070
    if seed % 4 == 3:  # a few huge terms among small ones
        lam[:, :3] *= 2.0 ** 900
    tgt = (rng.random(lam.shape) < 0.5).astype(np.uint8)
    got = oracle.objective_f64(lam, w, f, tgt)
    assert got == math.fsum(eq6_terms(lam, w, f, tgt))


def _one_chunk_sum(values):
    """A one-chunk instance whose terms are exactly `values`: every worker
    holds the chunk, demand 1, so requester r's term is its own w_r."""
    m = len(values)
    lam = np.ones((m, 1))
    w = np.array(values, dtype=np.float64).reshape(m, 1)
    f = np.zeros((m, m, 1))
    return oracle.objective_f64(lam, w, f, np.ones((m, 1), np.uint8))


def test_exact_sum_rounding_edges():
    u = 2.0 ** -53
    assert _one_chunk_sum([1.0, u]) == 1.0                 # tie: to even
    assert _one_chunk_sum([1.0 + 2 * u, u]) == 1.0 + 4 * u  # tie: to even (up)
    assert _one_chunk_sum([1.0, u, 2.0 ** -200]) == 1.0 + 2 * u  # just above the tie
    assert _one_chunk_sum([1.0] + [2.0 ** -60] * 200) == math.fsum([1.0] + [2.0 ** -60] * 200)
    tiny = 5e-324
    assert _one_chunk_sum([tiny] * 7) == 7 * tiny           # denormal, exact
    assert _one_chunk_sum([2.0 ** -1022 - tiny, tiny]) == 2.0 ** -1022  # into the normals
    big = 1.7976931348623157e308
    assert _one_chunk_sum([big, big]) == math.inf          # beyond the largest double
    # half an ulp (2^970) above the largest double is a tie, and its odd
    # mantissa rounds up, past the largest; less than that rounds down
    assert _one_chunk_sum([big, 2.0 ** 970]) == math.inf
    assert _one_chunk_sum([big, 2.0 ** 970 - 2.0 ** 917]) == big
    assert _one_chunk_sum([big, 2.0 ** 969]) == big
    assert _one_chunk_sum([0.0, 0.0]) == 0.0
    vals = [3.0 ** k * 2.0 ** -30 for k in range(40)] + [1e-300, 1e300, -0.0 + 0.0]
    assert _one_chunk_sum(vals) == math.fsum(vals)


def _exact_g(lam, w, f, tgt):
    return sum((Fraction(float(x)) for x in eq6_terms(lam, w, f, tgt)), Fraction(0))


def _algorithm1_exact(parent, lam, w, f, cap, order, eps, max_rounds=0):
    """Algorithm 1 for one start order, every acceptance decided on exact
    rationals: the exact G of the placement with worker h's set replaced
    must exceed the exact G of the current placement plus epsilon.  The
    update itself (marginals, rooted-tree DP) is the oracle's, pinned above."""
    m, n = lam.shape
    tgt = np.zeros((m, n), np.uint8)
    for h in order:
        p = oracle.marginal_f64(lam, w, f, tgt, h)
        tgt[h] = oracle.rooted_dp_f64(parent, p, int(cap[h]))[0]
    sweeps = accepts = ties = 0
    while True:
        improved = False
        for h in order:
            g_old = _exact_g(lam, w, f, tgt)
            old = tgt[h].copy()
            tgt[h] = 0
            p = oracle.marginal_f64(lam, w, f, tgt, h)
            tgt[h] = oracle.rooted_dp_f64(parent, p, int(cap[h]))[0]
            g_new = _exact_g(lam, w, f, tgt)
            if g_new > g_old + Fraction(eps):
                improved = True
                accepts += 1
            else:
                if g_new == g_old and not np.array_equal(old, tgt[h]):
                    ties += 1  # a different set of exactly equal value
                tgt[h] = old
        sweeps += 1
        if not improved or (max_rounds and sweeps == max_rounds):
            break
    return tgt, sweeps, accepts, float(_exact_g(lam, w, f, tgt)), ties


def test_acceptance_matches_exact_rational_driver():
    """Every decision equals the exact-rational one, at epsilon = 0 (where
    replacements of equal value must be rejected whatever the rounding of
    two sums would say) and at a small epsilon; some cases hit such ties."""
    ties = 0
    for seed in range(60):
        rng = np.random.default_rng(800 + seed)
        m = int(rng.integers(2, 6))
        n = int(rng.integers(5, 120))
        inst = W.random_instance(n, m, rng, kmax=int(rng.choice([3, 40, n + 2])),
                                 source_dependent=bool(seed % 4))
        lam, w, f = W.real_valued(inst, seed, jitter=0.5)
        order = [int(x) for x in rng.permutation(m)]
        eps = 0.0 if seed % 3 else 1e-7 * float(np.sum(lam * w))
        tgt, sweeps, accepts, obj, t = _algorithm1_exact(
            inst.parent, lam, w, f, inst.cap, order, eps)
        ties += t
        r = oracle.plan_f64(inst.parent, lam, w, f, inst.cap, epsilon=eps,
                            n_starts=1, orders_in=np.array([order], np.int32))
        assert r.start_sweeps.tolist() == [sweeps]
        assert r.start_accepts.tolist() == [accepts]
        np.testing.assert_array_equal(r.target, tgt)
        assert r.objective == obj
    assert ties > 0


@pytest.mark.parametrize("seed", range(30))
def test_proposition1_exact_gain_identity(seed):
    """G(T_-h with S as worker h's set) = G(T_-h) + sum_{b in S} p_h(b)."""
    parent, lam, w, f, cap = real_instance(seed, source_dependent=bool(seed % 2))
    rng = np.random.default_rng(50 + seed)
    m, n = lam.shape
    tgt = (rng.random((m, n)) < 0.4).astype(np.uint8)
    h = int(rng.integers(0, m))
    # p_h is defined with every worker but h fixed: h's own set is ignored
    p_own = oracle.marginal_f64(lam, w, f, tgt, h)
    tgt[h] = 0
    p = oracle.marginal_f64(lam, w, f, tgt, h)
    np.testing.assert_array_equal(p_own, p)
    g0 = oracle.objective_f64(lam, w, f, tgt)
    s = (rng.random(n) < 0.5).astype(np.uint8)
    tgt[h] = s
    g1 = oracle.objective_f64(lam, w, f, tgt)
    scale = max(g1, 1.0)
    assert g1 - g0 == pytest.approx(math.fsum(p[s == 1]), abs=1e-11 * scale)
    assert np.all(p >= 0.0)


# ------------------------------------------------------------ the planner

def _plans(inst_like, **kw):
    parent, lam, w, f, cap = inst_like
    a = oracle.plan(parent, lam, w, f, cap, **kw)
    b = oracle.plan_f64(parent, lam.astype(np.float64), w.astype(np.float64),
                        f.astype(np.float64), cap, epsilon=0.0, **kw)
    return a, b


def _same_as_integer(a, b):
    assert b.objective == float(a.objective)
    np.testing.assert_array_equal(b.target, a.target)
    np.testing.assert_array_equal(b.standalone, a.standalone.astype(np.float64))
    np.testing.assert_array_equal(b.orders, a.orders)
    np.testing.assert_array_equal(b.start_objective,
                                  a.start_objective.astype(np.float64))
    np.testing.assert_array_equal(b.start_sweeps, a.start_sweeps)
    np.testing.assert_array_equal(b.start_accepts, a.start_accepts)
    assert (b.best_start, b.updates, b.dp_cells) == (a.best_start, a.updates, a.dp_cells)


@pytest.mark.parametrize("seed", range(40))
def test_integer_valued_doubles_reproduce_the_integer_planner(seed):
    rng = np.random.default_rng(seed)
    m = int(rng.integers(1, 6))
    n = int(rng.integers(1, 120))
    inst = W.random_instance(n, m, rng, kmax=int(rng.choice([3, 30, n + 2])),
                             source_dependent=bool(seed % 3),
                             value_range=int(rng.choice([5, 100, 10 ** 5])))
    kw = dict(n_starts=int(rng.integers(0, 4)), max_rounds=int(rng.integers(0, 3)),
              order_seed=int(rng.integers(0, 2 ** 62)),
              flags=oracle.F_NO_REFINE if seed % 5 == 0 else 0)
    a, b = _plans((inst.parent, inst.demand, inst.recompute_cost,
                   inst.fetch_cost, inst.cap), **kw)
    _same_as_integer(a, b)


@pytest.mark.parametrize("name", ["tiny", "tree2k"])
def test_integer_valued_workloads_reproduce_the_integer_planner(name):
    inst = W.make_workload(name)
    kw = dict(n_starts=inst.n_starts, max_rounds=inst.max_rounds,
              order_seed=inst.order_seed)
    a, b = _plans((inst.parent, inst.demand, inst.recompute_cost,
                   inst.fetch_cost, inst.cap), **kw)
    _same_as_integer(a, b)


def joint_optimum_f64(parent, lam, w, f, cap):
    m, n = lam.shape
    sets = [np.array(bf.closed_sets(parent, int(cap[h]))) for h in range(m)]
    best = 0.0
    for combo in itertools.product(*[range(len(s)) for s in sets]):
        hold = np.stack([sets[h][combo[h]] for h in range(m)]).astype(np.uint8)
        best = max(best, objective_numpy(lam, w, f, hold))
    return best


@pytest.mark.parametrize("seed", range(25))
def test_theorem3_every_greedy_start_reaches_half(seed):
    parent, lam, w, f, cap = real_instance(2000 + seed, n_max=5, m_max=3)
    m = lam.shape[0]
    opt = joint_optimum_f64(parent, lam, w, f, cap)
    for order in itertools.permutations(range(m)):
        r = oracle.plan_f64(parent, lam, w, f, cap, n_starts=1,
                            orders_in=np.array([order], np.int32),
                            flags=oracle.F_NO_REFINE)
        assert r.objective >= 0.5 * opt * (1 - 1e-12)
        assert r.objective <= opt * (1 + 1e-12)


@pytest.mark.parametrize("seed", range(25))
def test_tolerance_gates_refinement(seed):
    parent, lam, w, f, cap = real_instance(3000 + seed)
    greedy = oracle.plan_f64(parent, lam, w, f, cap, n_starts=2,
                             flags=oracle.F_NO_REFINE)
    # an unreachable tolerance: one sweep, nothing accepted, greedy result
    frozen = oracle.plan_f64(parent, lam, w, f, cap, n_starts=2, epsilon=1e300)
    assert frozen.start_accepts.tolist() == [0, 0]
    assert frozen.start_sweeps.tolist() == [1, 1]
    np.testing.assert_array_equal(frozen.target, greedy.target)
    assert frozen.objective == greedy.objective
    # a finite tolerance: each accepted replacement raised G by more than it
    eps = 1e-3 * max(greedy.objective, 1.0)
    r = oracle.plan_f64(parent, lam, w, f, cap, n_starts=2, epsilon=eps)
    for s in range(2):
        gain = r.start_objective[s] - greedy.start_objective[s]
        assert gain >= r.start_accepts[s] * eps * (1 - 1e-9)
        assert r.start_objective[s] >= greedy.start_objective[s]


@pytest.mark.parametrize("seed", range(15))
def test_power_of_two_scaling_is_exact(seed):
    """Doubling Lambda (and epsilon) doubles every product and sum exactly:
    same decisions, objective exactly doubled."""
    parent, lam, w, f, cap = real_instance(4000 + seed)
    a = oracle.plan_f64(parent, lam, w, f, cap, n_starts=2, epsilon=1e-6)
    b = oracle.plan_f64(parent, 2.0 * lam, w, f, cap, n_starts=2, epsilon=2e-6)
    np.testing.assert_array_equal(a.target, b.target)
    assert b.objective == 2.0 * a.objective
    np.testing.assert_array_equal(b.start_objective, 2.0 * a.start_objective)


def test_invalid_real_inputs_are_rejected():
    parent, lam, w, f, cap = real_instance(7, n_max=10)
    for bad in (np.nan, np.inf, -1.0):
        l2 = lam.copy()
        l2[0, 0] = bad
        with pytest.raises(oracle.OracleError):
            oracle.plan_f64(parent, l2, w, f, cap)
        f2 = f.copy()
        f2[0, 0, 0] = bad
        with pytest.raises(oracle.OracleError):
            oracle.plan_f64(parent, lam, w, f2, cap)
    with pytest.raises(oracle.OracleError):
        oracle.plan_f64(parent, lam, w, f, cap, epsilon=-1.0)


@pytest.mark.parametrize("seed", range(30))
def test_safeguards_on_integer_valued_doubles_match_integer(seed):
    """Requester-side inputs with the comparator safeguards: the real-valued
    planner on integer-valued doubles reproduces the integer planner's
    candidates and choice exactly (all sums exact)."""
    rng = np.random.default_rng(600 + seed)
    m = int(rng.integers(1, 5))
    n = int(rng.integers(1, 80))
    inst = W.random_instance(n, m, rng, kmax=int(rng.choice([3, 20, n + 2])),
                             source_dependent=False,
                             value_range=int(rng.choice([5, 100])))
    flags = oracle.F_SAFEGUARDS | (oracle.F_NO_REFINE if seed % 2 else 0)
    a = oracle.plan(inst.parent, inst.demand, inst.recompute_cost,
                    inst.fetch_cost, inst.cap, n_starts=1, flags=flags)
    b = oracle.plan_f64(inst.parent, inst.demand.astype(float),
                        inst.recompute_cost.astype(float),
                        inst.fetch_cost.astype(float), inst.cap, n_starts=1,
                        flags=flags)
    assert a.safeguards_run and b.safeguards_run
    assert b.safeguard_objective == tuple(float(x) for x in a.safeguard_objective)
    assert (b.best_start, b.updates, b.dp_cells) == (a.best_start, a.updates, a.dp_cells)
    assert b.objective == float(a.objective)
    np.testing.assert_array_equal(b.target, a.target)


def test_safeguards_real_values_and_signed_zero():
    """On real requester-side costs the candidates run, the returned plan is
    the argmax of the starts and the candidates, and a fetch plane whose
    sources differ only by the sign of a zero still counts as
    requester-side."""
    parent, lam, w, f, cap = real_instance(5, n_max=40, m_max=3,
                                           source_dependent=False)
    m = lam.shape[0]
    f[f == f.min()] = 0.0
    if m > 2:
        g = f.copy()
        g[1, 2][g[1, 2] == 0.0] = -0.0  # -0.0 == 0.0 as values
        f = g
    plain = oracle.plan_f64(parent, lam, w, f, cap, n_starts=1)
    sg = oracle.plan_f64(parent, lam, w, f, cap, n_starts=1,
                         flags=oracle.F_SAFEGUARDS)
    assert sg.safeguards_run
    assert sg.objective == max([plain.objective] + list(sg.safeguard_objective))
    src = f.copy()
    if m > 2:
        src[0, m - 1, 0] += 1.0  # one source differs: not requester-side
        nd = oracle.plan_f64(parent, lam, w, src, cap, n_starts=1,
                             flags=oracle.F_SAFEGUARDS)
        assert not nd.safeguards_run
