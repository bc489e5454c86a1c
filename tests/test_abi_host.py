"""Boundary checks that need no GPU: the C-ABI library loads, exports every
function include/prefixplace.h declares, and validates inputs (through
PP_F_VALIDATE_ONLY) before any device work."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2608_01655_amd import binding as B
from paper_2608_01655_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(B.LIB_PATH):
        from paper_2608_01655_amd import build

        build.build()
    return B.lib()


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "prefixplace.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"\b(pp_[a-z_]+)\s*\(", src)
    return sorted(set(names))


def test_every_declared_symbol_is_exported(L):
    names = _declared_functions()
    assert "pp_plan" in names and "pp_rooted_dp" in names
    assert len(names) >= 11
    for name in names:
        assert hasattr(L, name), name
    assert B.pp_abi_version() == 11


def _validate(inst, **kw):
    args = dict(n_starts=inst.n_starts, max_rounds=inst.max_rounds,
                order_seed=inst.order_seed, flags=B.PP_F_VALIDATE_ONLY)
    args.update(kw)
    return B.pp_plan(inst.parent, inst.demand, inst.recompute_cost,
                     inst.fetch_cost, inst.cap, **args)


def test_validate_only_accepts_good_input(L):
    inst = W.make_workload("tiny")
    p = _validate(inst)
    assert p.target.sum() == 0  # outputs untouched


def _expect(code, fn):
    with pytest.raises(B.PPError) as e:
        fn()
    assert e.value.code == code
    assert B.pp_last_error()


def test_validation_errors(L):
    rng = np.random.default_rng(0)
    inst = W.random_instance(10, 3, rng)
    bad = inst.parent.copy()
    bad[3] = 3
    _expect(B.PP_E_TREE, lambda: B.pp_plan(bad, inst.demand, inst.recompute_cost,
                                           inst.fetch_cost, inst.cap,
                                           flags=B.PP_F_VALIDATE_ONLY))
    cyc = np.array([1, 2, 0, -1, -1, -1, -1, -1, -1, -1], np.int32)
    _expect(B.PP_E_TREE, lambda: B.pp_plan(cyc, inst.demand, inst.recompute_cost,
                                           inst.fetch_cost, inst.cap,
                                           flags=B.PP_F_VALIDATE_ONLY))
    oob = inst.parent.copy()
    oob[5] = 10
    _expect(B.PP_E_TREE, lambda: _validate_with(inst, parent=oob))
    d = inst.demand.copy()
    d[1, 1] = -1
    _expect(B.PP_E_RANGE, lambda: _validate_with(inst, demand=d))
    f = inst.fetch_cost.copy()
    f[2, 0, 4] = -3
    _expect(B.PP_E_RANGE, lambda: _validate_with(inst, fetch=f))
    c = inst.cap.copy()
    c[0] = -1
    _expect(B.PP_E_RANGE, lambda: _validate_with(inst, cap=c))
    big = np.full_like(inst.demand, 2 ** 31)
    _expect(B.PP_E_OVERFLOW, lambda: _validate_with(inst, demand=big, w=big))
    _expect(B.PP_E_ARG, lambda: _validate(inst, n_starts=-1))
    _expect(B.PP_E_ARG, lambda: _validate(inst, n_starts=1,
                                          orders=np.array([[0, 1, 1]], np.int32)))
    _expect(B.PP_E_ARG, lambda: _validate(inst, n_starts=0,
                                          orders=np.array([[0, 1, 2]], np.int32)))


def _validate_with(inst, parent=None, demand=None, w=None, fetch=None, cap=None):
    return B.pp_plan(inst.parent if parent is None else parent,
                     inst.demand if demand is None else demand,
                     inst.recompute_cost if w is None else w,
                     inst.fetch_cost if fetch is None else fetch,
                     inst.cap if cap is None else cap,
                     flags=B.PP_F_VALIDATE_ONLY)


def test_bad_sizes_rejected(L):
    P = ctypes.c_void_p
    z = np.zeros(4, np.int64)
    for n, m in ((0, 1), (1, 0), (1, 256)):
        rc = L.pp_plan(n, m, z.ctypes.data_as(P), z.ctypes.data_as(P),
                       z.ctypes.data_as(P), z.ctypes.data_as(P),
                       z.ctypes.data_as(P), None, z.ctypes.data_as(P),
                       z.ctypes.data_as(P), None)
        assert rc == B.PP_E_ARG
    rc = L.pp_plan(1, 1, None, None, None, None, None, None, None, None, None)
    assert rc == B.PP_E_ARG


def test_orders_match_oracle(L, oracle_mod):
    rng = np.random.default_rng(5)
    for m in (1, 2, 3, 5, 6, 9, 16):
        st = rng.integers(0, 5, size=m).astype(np.int64)  # ties
        for S in (0, 1, 2, 8, 11):
            seed = int(rng.integers(0, 2 ** 63))
            assert B.pp_num_starts(m, S) == oracle_mod.num_starts(m, S)
            np.testing.assert_array_equal(B.pp_orders(m, S, seed, st),
                                          oracle_mod.orders(m, S, seed, st))


def test_replan_validation(L):
    inst = W.make_workload("tiny")
    inc = np.zeros((inst.m, inst.n), np.uint8)

    def call(incumbent=inc, horizon=1):
        return B.pp_replan(inst.parent, inst.demand, inst.recompute_cost,
                           inst.fetch_cost, inst.cap, incumbent, horizon,
                           flags=B.PP_F_VALIDATE_ONLY)

    r = call()
    assert r.target.sum() == 0 and not r.adopt  # outputs untouched
    _expect(B.PP_E_ARG, lambda: call(horizon=-1))
    two = inc.copy()
    two[0, 0] = 2
    _expect(B.PP_E_ARG, lambda: call(incumbent=two))
    bad = inst.parent.copy()
    bad[1] = 1
    _expect(B.PP_E_TREE, lambda: B.pp_replan(
        bad, inst.demand, inst.recompute_cost, inst.fetch_cost, inst.cap, inc,
        1, flags=B.PP_F_VALIDATE_ONLY))
    P = ctypes.c_void_p
    z = np.zeros(64, np.int64)
    info = B.pp_replan_info()
    rc = L.pp_replan(2, 1, z.ctypes.data_as(P), z.ctypes.data_as(P),
                     z.ctypes.data_as(P), z.ctypes.data_as(P),
                     z.ctypes.data_as(P), z.ctypes.data_as(P), 1, None,
                     z.ctypes.data_as(P), None, None, None)
    assert rc == B.PP_E_ARG  # info is required


def test_real_valued_validation(L):
    inst = W.make_workload("tiny")
    lam, w, f = (inst.demand.astype(float), inst.recompute_cost.astype(float),
                 inst.fetch_cost.astype(float))

    def call(lam=lam, w=w, f=f, eps=0.0, flags=B.PP_F_VALIDATE_ONLY):
        return B.pp_plan_f64(inst.parent, lam, w, f, inst.cap, epsilon=eps,
                             flags=flags)

    p = call()
    assert p.target.sum() == 0
    for bad in (np.nan, np.inf, -0.5):
        l2 = lam.copy()
        l2[1, 2] = bad
        _expect(B.PP_E_RANGE, lambda: call(lam=l2))
        f2 = f.copy()
        f2[0, 1, 3] = bad
        _expect(B.PP_E_RANGE, lambda: call(f=f2))
    _expect(B.PP_E_ARG, lambda: call(eps=-1.0))
    _expect(B.PP_E_ARG, lambda: call(eps=np.nan))
    call(flags=B.PP_F_VALIDATE_ONLY | B.PP_F_SAFEGUARDS)  # offered
    _expect(B.PP_E_RANGE, lambda: B.pp_rooted_dp_f64(inst.parent,
                                                     np.full(inst.n, -1.0), 3))


def _caterpillar(depth):
    """Spine 0..depth-1 plus one leaf per spine node; the spine child has the
    smaller id, so every leaf's row stays pending while the spine below it
    is swept (one pending skip target per level)."""
    parent = [-1] + list(range(0, depth - 1)) + list(range(0, depth))
    return np.array(parent, np.int32)


def test_pending_skip_rows_beyond_the_lds_slots(L):
    """Up to 254 pending skip rows stay in LDS slots; deeper trees spill the
    long-lived ones to device memory instead of failing."""
    for depth, spills in ((250, False), (300, True), (1000, True), (5000, True)):
        parent = _caterpillar(depth)
        n = parent.shape[0]
        lam = np.ones((1, n), np.int64)
        w = np.ones((1, n), np.int64)
        f = np.zeros((1, 1, n), np.int64)
        B.pp_plan(parent, lam, w, f, np.array([5], np.int32), n_starts=1,
                  flags=B.PP_F_VALIDATE_ONLY)
        meta, slots = B.pp_sweep_layout(parent, 1)
        nspill = B.pp_sweep_spills(parent)[0]
        assert (nspill > 0) == spills
        assert slots <= 254 and (not spills or slots < 100)
