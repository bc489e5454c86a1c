"""CPU check of the DP sweep's step schedule (no GPU).

The library exports, per tree, the metadata its gfx950 sweep follows: which
steps are leaves (a lane mask: their skip operand is the previous row, in
registers), which LDS row each row is stored to (a slot if a later row
skips to it, else one of a few sink rows), and which slot each other step's
skip operand is read from.  This test replays that schedule on whole DP
rows with numpy, in the kernel's order -- a step stores its row, then reads
the skip row of the step two ahead; after each group of sink-row-count
steps the rows of those steps must still be in place for the gather of the
stage's last column -- and
requires the replay to reproduce the oracle's rooted-tree optimum and
selection (Eq. 9, Theorem 1, tie rule R1).  A wrong slot, a slot reused too
early, or a read issued too early gives a different value or set, or fails
the gather check.
"""

import numpy as np
import pytest

from paper_2608_01655_amd import binding as B
from paper_2608_01655_amd import workloads as W
from tests import bruteforce as bf

BATCH = 32




def replay(parent, profit, k, cells):
    meta, slots = B.pp_sweep_layout(parent, cells)
    nspill, outs, ins = B.pp_sweep_spills(parent)
    spill = {}                                   # spill index -> row values
    n = len(parent)
    kk = min(k, n)
    order = bf.canonical_preorder(parent)
    nsteps = meta.shape[0]
    assert nsteps % BATCH == 0 and nsteps - n < BATCH
    pad = nsteps - n
    row = 64 * cells * 8 + 8                     # LDS row stride (bytes)
    sink = 16 if cells == 1 else 4               # sink rows = gather group
    zero = slots                                 # slots | zero | sink rows
    rows = np.zeros((slots + 1 + sink, kk + 1), dtype=object)
    x = np.zeros(kk + 1, dtype=object)
    pre = [np.zeros(kk + 1, dtype=object) for _ in range(2)]
    bits = np.zeros((nsteps, kk + 1), dtype=bool)
    group = []                                   # (row, value) of this group
    for s in range(nsteps):
        if s % BATCH == 0 and nspill:
            # at a batch boundary B: the copy-outs of batch B-2 at the latest
            # (they precede the staging of batch B), the copy-ins of batch
            # B+1 at the earliest (once batch B-1 is done)
            b = s // BATCH
            if b >= 2:
                for ts, sx in outs[b - 2]:
                    spill[int(sx)] = rows[int(ts)].copy()
            for bb in ([0, 1] if b == 0 else [b + 1]):
                if bb < len(ins):
                    for rs, sx in ins[bb]:
                        assert int(rs) != zero
                        rows[int(rs)] = spill[int(sx)].copy()
        st, pf, m2, m3 = (int(v) for v in meta[s])
        assert m2 in (0, 0xFFFFFFFF) and m3 == 0
        leaf = m2 != 0
        if s == 0:
            assert leaf                           # padded step 0 is a leaf
        assert pf % row == 0 and pf // row <= zero
        assert st % row == 0 and st // row != zero and st // row <= zero + sink
        sk = x if leaf else pre[s % 2]
        p = int(profit[order[n - 1 - (s - pad)]]) if s >= pad else 0
        t = np.empty(kk + 1, dtype=object)
        t[0] = -1
        t[1:] = x[:-1] + p
        take = t > sk
        take[0] = False
        y = np.where(take, t, sk)
        y[0] = 0
        bits[s] = take
        rows[st // row] = y                      # its slot, or a sink row
        group.append((st // row, y))
        assert all(v == 0 for v in rows[zero])   # the zero row stays zero
        # after the store: the skip row of step s+2 (word 1 of step s+1)
        nxt = int(meta[s + 1][1]) if s + 1 < nsteps else zero * row
        pre[s % 2] = rows[nxt // row].copy()
        if s % sink == sink - 1:                 # the gather of the group:
            for r_, v in group:                  # every row still in place
                assert list(rows[r_]) == list(v)
            group = []
        x = y
    # backtrack over the recorded choice bits, in preorder positions
    nextpos = np.empty(n, np.int64)
    pos_of = {v: i for i, v in enumerate(order)}
    size = np.ones(n, np.int64)
    for v in reversed(order):
        if parent[v] >= 0:
            size[pos_of[parent[v]]] += size[pos_of[v]]
    nextpos[:] = np.arange(n) + size
    sel = np.zeros(n, np.uint8)
    q, j = 0, kk
    while q < n and j > 0:
        if bits[n - 1 - q + pad][j]:
            sel[order[q]] = 1
            q, j = q + 1, j - 1
        else:
            q = int(nextpos[q])
    return int(x[kk]) if kk > 0 else 0, sel


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import os

    if not os.path.exists(B.LIB_PATH):
        from paper_2608_01655_amd import build

        build.build()


@pytest.mark.parametrize("seed", range(40))
def test_replayed_schedule_matches_oracle(oracle_mod, seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 260))
    parent = W.random_forest(n, rng, p_root=float(rng.choice([0.0, 0.1, 0.4])))
    profit = rng.integers(0, int(rng.choice([3, 50, 10 ** 6])), size=n)
    k = int(rng.integers(0, n + 3))
    cells = int(rng.choice([1, 2, 4]))
    val, sel = replay(parent, profit, k, cells)
    osel, oval = oracle_mod.rooted_dp(parent, profit, k)
    assert val == oval
    np.testing.assert_array_equal(sel, osel)


def test_replayed_schedule_deep_and_wide(oracle_mod):
    rng = np.random.default_rng(9)
    comb = np.array([-1] + list(range(0, 199)) + list(range(0, 200)), np.int32)
    path = np.arange(-1, 299, dtype=np.int32)
    star = np.array([-1] + [0] * 299, np.int32)
    for parent in (comb, path, star):
        profit = rng.integers(0, 20, size=parent.shape[0])
        for k in (1, 70, parent.shape[0]):
            val, sel = replay(parent, profit, k, 2)
            osel, oval = oracle_mod.rooted_dp(parent, profit, k)
            assert val == oval
            np.testing.assert_array_equal(sel, osel)


caterpillar = W.caterpillar
conversation_tree = W.regenerated_conversation


@pytest.mark.parametrize("depth", [256, 300, 700])
def test_replayed_schedule_with_spilled_rows(oracle_mod, depth):
    """More pending skip rows than the LDS slots hold: long-lived rows are
    spilled to device memory and restored; the replay, with every copy-out at
    its latest and every copy-in at its earliest time, must still give the
    oracle's optimum and set."""
    parent = caterpillar(depth)
    nspill, outs, ins = B.pp_sweep_spills(parent)
    assert nspill > 0
    meta, slots = B.pp_sweep_layout(parent, 1)
    assert slots < 254
    rng = np.random.default_rng(depth)
    n = parent.shape[0]
    for k in (1, 64, 300, n):
        profit = rng.integers(0, 30, size=n)
        for cells in (1, 2):
            val, sel = replay(parent, profit, k, cells)
            osel, oval = oracle_mod.rooted_dp(parent, profit, k)
            assert val == oval
            np.testing.assert_array_equal(sel, osel)


@pytest.mark.parametrize("seed", range(6))
def test_replayed_schedule_branching_chains(oracle_mod, seed):
    rng = np.random.default_rng(77 + seed)
    parent = conversation_tree(int(rng.integers(1500, 4000)), rng)
    assert B.pp_sweep_spills(parent)[0] > 0
    perm = rng.permutation(parent.shape[0]) if seed % 2 else None
    if perm is not None:  # relabel: the schedule follows the canonical preorder
        inv = np.empty_like(perm)
        inv[perm] = np.arange(perm.shape[0])
        parent = np.array([-1 if parent[perm[v]] < 0 else inv[parent[perm[v]]]
                           for v in range(parent.shape[0])], np.int32)
    profit = rng.integers(0, 1000, size=parent.shape[0])
    k = int(rng.choice([100, 1000]))
    val, sel = replay(parent, profit, k, 1)
    osel, oval = oracle_mod.rooted_dp(parent, profit, k)
    assert val == oval
    np.testing.assert_array_equal(sel, osel)


def test_layout_of_benchmark_trees():
    """Stack depth of the benchmark trees stays small (LDS-resident)."""
    for name, limit in (("tree50k", 20), ("chat50k", 24), ("rag10k", 16)):
        inst = W.make_workload(name)
        meta, slots = B.pp_sweep_layout(inst.parent, 2)
        assert slots <= limit
        assert B.pp_sweep_spills(inst.parent)[0] == 0  # nothing spilled
        assert meta.shape[0] == (inst.n + 31) // 32 * 32
