"""Seeded synthetic inputs for the prefix-placement planner.

This module only *draws* inputs: prefix trees, per-worker demand, recompute
costs and pairwise fetch costs, all as integers (demand in requests per epoch,
costs in microseconds).  It holds none of the planner's arithmetic (no savings,
marginals, DP or objective), so both the HIP path and the CPU oracle can read
the same inputs without sharing method code.

Shapes follow the workloads the paper describes (Section V-A): a RAG-shaped
tree with a shared system prompt and document branches, multi-turn
conversation chains, Zipf-skewed leaf popularity split across workers with a
shared-request fraction, requester hardware factors in the ratios of the
profiled T4/L4/A100 GPUs, and fetch costs derived from the KV footprint of a
512-token chunk (36,864 bytes per token, Table 1) over an effective goodput in
Gb/s (Eq. 1).  The paper's datasets are not used; these synthetic inputs
stand in for them.
"""

from __future__ import annotations

import dataclasses
from collections import deque

import numpy as np

# 36,864 bytes per token (3B model, FP16; Table 1) times a 512-token chunk.
CHUNK_BYTES = 36_864 * 512
# Fetch microseconds for a chunk at `bw` Gb/s is CHUNK_BITS_US_NUM / (1000 * bw).
CHUNK_BITS_US_NUM = CHUNK_BYTES * 8  # bits; divided by Gb/s * 1000 gives us

# Depth-linear materialisation cost a + b*depth, in microseconds, scaled by a
# per-worker hardware factor h.  Factors are stored as h10 = 10*h so that
# h10 * (a + b*d) / 10 is an exact integer for the factors used here.
COST_A_US = 20_000
COST_B_US = 6_000


@dataclasses.dataclass
class Instance:
    """One planner input, with node ids already in canonical preorder."""

    name: str
    parent: np.ndarray          # int32 [n]; -1 marks a child of the dummy root
    demand: np.ndarray          # int64 [m][n]
    recompute_cost: np.ndarray  # int64 [m][n]
    fetch_cost: np.ndarray      # int64 [m][m][n]; [src][dst][b]
    cap: np.ndarray             # int32 [m]
    n_starts: int
    max_rounds: int
    order_seed: int
    depth: np.ndarray           # int32 [n], root depth 0 (generator metadata)

    @property
    def n(self) -> int:
        return int(self.parent.shape[0])

    @property
    def m(self) -> int:
        return int(self.demand.shape[0])

    def checksum(self) -> str:
        import hashlib

        h = hashlib.sha256()
        for a in (self.parent, self.demand, self.recompute_cost,
                  self.fetch_cost, self.cap):
            h.update(np.ascontiguousarray(a).tobytes())
        h.update(f"{self.n_starts},{self.max_rounds},{self.order_seed}".encode())
        return h.hexdigest()


# --------------------------------------------------------------------------
# Trees
# --------------------------------------------------------------------------

def _relabel_preorder(par: list[int]) -> tuple[np.ndarray, np.ndarray]:
    """Relabel a rooted forest (parent list, -1 = root) into canonical preorder:
    roots in increasing id, children in increasing id.  Returns (parent, perm)
    where perm[old] = new."""
    n = len(par)
    children: list[list[int]] = [[] for _ in range(n)]
    roots = []
    for v in range(n):
        if par[v] < 0:
            roots.append(v)
        else:
            children[par[v]].append(v)
    perm = np.empty(n, dtype=np.int64)
    pos = 0
    stack = list(reversed(roots))
    while stack:
        v = stack.pop()
        perm[v] = pos
        pos += 1
        stack.extend(reversed(children[v]))
    new_parent = np.full(n, -1, dtype=np.int32)
    for v in range(n):
        if par[v] >= 0:
            new_parent[perm[v]] = perm[par[v]]
    return new_parent, perm


def _depths(parent: np.ndarray) -> np.ndarray:
    """Depth of each node of a preorder-labelled forest (parent[v] < v)."""
    d = np.zeros(parent.shape[0], dtype=np.int32)
    for v in range(parent.shape[0]):
        p = parent[v]
        if p >= 0:
            d[v] = d[p] + 1
    return d


def galton_watson_tree(n: int, lam: float, dmax: int,
                       rng: np.random.Generator) -> list[int]:
    """Grow a tree breadth-first: each popped node below depth `dmax` gets
    Poisson(lam) children.  When the queue runs dry before n nodes exist, a
    new round re-enqueues every node shallower than `dmax` in id order."""
    par = [-1]
    depth = [0]
    q = deque([0])
    while len(par) < n:
        if not q:
            q.extend(v for v in range(len(par)) if depth[v] < dmax)
        v = q.popleft()
        if depth[v] >= dmax:
            continue
        c = int(rng.poisson(lam))
        c = min(c, n - len(par))
        for _ in range(c):
            par.append(v)
            depth.append(depth[v] + 1)
            q.append(len(par) - 1)
    return par


def rag_tree(n: int, n_templates: int, rng: np.random.Generator) -> list[int]:
    """Shared system prompt (root) -> template children -> retrieved-document
    subtrees.  Template t allows D_t ~ U{2..6} levels below it; nodes above
    that cap draw Geometric(1/3) children (mean 3).  Rounds refill as in
    `galton_watson_tree`."""
    par = [-1]
    depth = [0]
    cap = [0]  # absolute depth cap of the node's template
    q: deque[int] = deque()
    for _ in range(min(n_templates, n - 1)):
        par.append(0)
        depth.append(1)
        cap.append(1 + int(rng.integers(2, 7)))
        q.append(len(par) - 1)
    while len(par) < n:
        if not q:
            q.extend(v for v in range(1, len(par)) if depth[v] < cap[v])
        v = q.popleft()
        if depth[v] >= cap[v]:
            continue
        c = int(rng.geometric(1.0 / 3.0))
        c = min(c, n - len(par))
        for _ in range(c):
            par.append(v)
            depth.append(depth[v] + 1)
            cap.append(cap[v])
            q.append(len(par) - 1)
    return par


def chain_tree(n: int, n_base: int, lam: float, dmax: int, dchain: int,
               rng: np.random.Generator) -> list[int]:
    """Conversation-shaped tree: a Galton-Watson base of `n_base` nodes, then
    single-child chains (length U{8..48}, capped at depth `dchain`) appended
    to uniformly chosen leaves of depth <= dchain-8 until n nodes exist."""
    par = galton_watson_tree(n_base, lam, dmax, rng)
    depth = [0] * len(par)
    nchild = [0] * len(par)
    for v in range(1, len(par)):
        depth[v] = depth[par[v]] + 1
        nchild[par[v]] += 1
    leaves = [v for v in range(len(par)) if nchild[v] == 0 and depth[v] <= dchain - 8]
    while len(par) < n:
        if not leaves:
            raise ValueError("no leaf left to extend")
        idx = int(rng.integers(0, len(leaves)))
        u = leaves[idx]
        length = int(rng.integers(8, 49))
        length = min(length, dchain - depth[u], n - len(par))
        # u stops being a leaf; the chain tip becomes one
        leaves[idx] = leaves[-1]
        leaves.pop()
        prev = u
        for _ in range(length):
            par.append(prev)
            depth.append(depth[prev] + 1)
            nchild.append(0)
            prev = len(par) - 1
        if depth[prev] <= dchain - 8:
            leaves.append(prev)
    return par


# --------------------------------------------------------------------------
# Demand and costs
# --------------------------------------------------------------------------

def zipf_leaf_demand(parent: np.ndarray, m: int, s: float, total: int,
                     rng: np.random.Generator, shared_num: int = 1,
                     shared_den: int = 2) -> np.ndarray:
    """Per-worker demand [m][n].  Leaf popularity is Zipf(s) over a random
    ranking; integer counts sum exactly to `total` (floor, then largest
    remainder, ties by leaf id).  Each leaf has a random home worker; a
    shared_num/shared_den share of its requests (rounded down) is spread
    evenly over all workers, the leftover units going one each to home+1,
    home+2, ... (mod m), and the rest stays at home.  A request counts at every chunk on its path, so
    a node's demand is the sum over the leaves below it."""
    n = parent.shape[0]
    has_child = np.zeros(n, dtype=bool)
    has_child[parent[parent >= 0]] = True
    leaves = np.flatnonzero(~has_child)
    nl = leaves.shape[0]
    rank = rng.permutation(nl) + 1
    wgt = rank.astype(np.float64) ** (-s)
    raw = total * wgt / wgt.sum()
    cnt = np.floor(raw).astype(np.int64)
    rem = total - int(cnt.sum())
    if rem > 0:
        frac = raw - cnt
        # largest remainder first, ties by leaf id (stable sort on -frac)
        order = np.argsort(-frac, kind="stable")
        cnt[order[:rem]] += 1
    home = rng.integers(0, m, size=nl)
    lam = np.zeros((m, n), dtype=np.int64)
    shared = (cnt * shared_num) // shared_den
    each = shared // m
    extra = shared % m
    lam[:, leaves] += each[None, :]
    for li in range(nl):
        e = int(extra[li])
        h = int(home[li])
        for t in range(1, e + 1):
            lam[(h + t) % m, leaves[li]] += 1
    lam[home, leaves] += cnt - shared
    # propagate to ancestors (children carry larger preorder ids)
    for v in range(n - 1, 0, -1):
        p = parent[v]
        if p >= 0:
            lam[:, p] += lam[:, v]
    return lam


def depth_linear_recompute(depth: np.ndarray, h10: np.ndarray) -> np.ndarray:
    """w[m][v] = h_m * (a + b*depth(v)) microseconds, exact in integers."""
    base = COST_A_US + COST_B_US * depth.astype(np.int64)
    w = h10.astype(np.int64)[:, None] * base[None, :]
    assert np.all(w % 10 == 0)
    return w // 10


def fetch_us_for_gbps(bw_gbps: np.ndarray) -> np.ndarray:
    """Microseconds to move one 512-token chunk at `bw_gbps` (Eq. 1:
    bytes / goodput), rounded half up."""
    return np.floor(CHUNK_BITS_US_NUM / (1000.0 * np.asarray(bw_gbps)) + 0.5
                    ).astype(np.int64)


def pairwise_fetch(m: int, n: int, lo: float, hi: float,
                   rng: np.random.Generator) -> np.ndarray:
    """fetch[src][dst][b]: an asymmetric goodput matrix, one independent
    U[lo, hi] Gb/s draw per ordered pair; chunks are equal-sized so the cost
    is the same for every b.  The diagonal is 0 (a worker never fetches from
    itself)."""
    bw = rng.uniform(lo, hi, size=(m, m))
    us = fetch_us_for_gbps(bw)
    np.fill_diagonal(us, 0)
    return np.ascontiguousarray(np.broadcast_to(us[:, :, None], (m, m, n))
                                .astype(np.int64))


def requester_fetch(m: int, n: int, us: int) -> np.ndarray:
    """Requester-side cost: the same value for every source != requester."""
    f = np.full((m, m, n), us, dtype=np.int64)
    for i in range(m):
        f[i, i, :] = 0
    return f


def _own_demand(parent: np.ndarray, demand: np.ndarray) -> np.ndarray:
    """Requests that end at each node: its demand minus its children's."""
    own = demand.copy()
    for v in range(parent.shape[0] - 1, 0, -1):
        p = parent[v]
        if p >= 0:
            own[:, p] -= demand[:, v]
    return own


def _aggregate(parent: np.ndarray, own: np.ndarray) -> np.ndarray:
    lam = own.copy()
    for v in range(parent.shape[0] - 1, 0, -1):
        p = parent[v]
        if p >= 0:
            lam[:, p] += lam[:, v]
    return lam


def shift_routing(parent: np.ndarray, demand: np.ndarray, num: int,
                  den: int) -> np.ndarray:
    """A routing shift between epochs: at every node, num/den of the requests
    that end there on worker m (rounded down) move to worker (m + 1) mod M;
    the demand is then re-aggregated along prefix paths.  num = den moves
    all routing mass.  `parent` must be preorder-labelled."""
    own = _own_demand(parent, demand)
    assert np.all(own >= 0), "demand is not aggregated along prefix paths"
    moved = (own * num) // den
    out = own - moved + np.roll(moved, 1, axis=0)
    return _aggregate(parent, out)


def perturb_popularity(parent: np.ndarray, demand: np.ndarray, sigma: float,
                       rng: np.random.Generator) -> np.ndarray:
    """A popularity perturbation between epochs: the requests ending at each
    node are scaled by one log-normal factor exp(sigma Z) per node (shared by
    all workers), rounded half up, then re-aggregated along prefix paths."""
    own = _own_demand(parent, demand)
    assert np.all(own >= 0), "demand is not aggregated along prefix paths"
    z = np.exp(sigma * rng.standard_normal(parent.shape[0]))
    out = np.floor(own * z[None, :] + 0.5).astype(np.int64)
    return _aggregate(parent, out)


def prefix_incumbent(n: int, cap: np.ndarray) -> np.ndarray:
    """A simple resident state for re-planning tests: worker h holds the
    first min(cap[h], n) nodes in preorder (a prefix of the preorder is
    closed under parents)."""
    inc = np.zeros((cap.shape[0], n), dtype=np.uint8)
    for h, k in enumerate(cap):
        inc[h, :min(int(k), n)] = 1
    return inc


def real_valued(inst: "Instance", seed: int, jitter: float = 0.25) -> tuple:
    """The workload in the paper's own units, as doubles: demand in requests
    per epoch scaled by a per-entry factor U[1 - jitter, 1 + jitter], and
    recompute and fetch costs in milliseconds (microseconds / 1000), each
    scaled by its own factor from the same range.  Returns (demand,
    recompute_cost, fetch_cost); the diagonal of the fetch plane stays 0."""
    rng = np.random.default_rng(seed)
    lo, hi = 1.0 - jitter, 1.0 + jitter
    lam = inst.demand * rng.uniform(lo, hi, size=inst.demand.shape)
    w = inst.recompute_cost / 1000.0 * rng.uniform(lo, hi, size=inst.recompute_cost.shape)
    f = inst.fetch_cost / 1000.0 * rng.uniform(lo, hi, size=inst.fetch_cost.shape)
    for i in range(inst.m):
        f[i, i, :] = 0.0
    return lam, w, f


# --------------------------------------------------------------------------
# The five benchmark workloads
# --------------------------------------------------------------------------

H10_CYCLE = np.array([6, 10, 25])  # 0.6 / 1.0 / 2.5 (A100 / L4 / T4-like ratios)

WORKLOADS = ("tiny", "tree2k", "rag10k", "tree50k", "chat50k")


def make_workload(name: str) -> Instance:
    """Build one of the five named workloads; the generator seed is the
    workload's 1-based index and so is the start-order seed."""
    idx = WORKLOADS.index(name) + 1
    rng = np.random.default_rng(idx)
    if name == "tiny":
        par = galton_watson_tree(200, 1.5, 8, rng)
        m, caps = 2, [40, 40]
        zipf_s, total = 1.1, 10_000
        h10 = np.array([10, 25])
        starts, rounds = 1, 3
    elif name == "tree2k":
        par = galton_watson_tree(2_000, 2.0, 12, rng)
        m, caps = 4, [256] * 4
        zipf_s, total = 1.0, 10 ** 6
        h10 = np.array([10, 10, 25, 6])
        starts, rounds = 4, 0
    elif name == "rag10k":
        par = rag_tree(10_000, 40, rng)
        m, caps = 8, [1_024] * 8
        zipf_s, total = 0.9, 10 ** 7
        h10 = H10_CYCLE[np.arange(8) % 3]
        starts, rounds = 8, 0
    elif name == "tree50k":
        par = galton_watson_tree(50_000, 2.2, 16, rng)
        m, caps = 16, [4_096] * 16
        zipf_s, total = 1.0, 10 ** 8
        h10 = H10_CYCLE[np.arange(16) % 3]
        starts, rounds = 8, 0
    elif name == "chat50k":
        par = chain_tree(50_000, 35_000, 2.2, 16, 64, rng)
        m = 16
        caps = [int(x) for x in rng.integers(2_048, 8_193, size=16)]
        zipf_s, total = 1.2, 10 ** 8
        h10 = H10_CYCLE[np.arange(16) % 3]
        starts, rounds = 32, 0
    else:
        raise KeyError(name)
    parent, _ = _relabel_preorder(par)
    n = parent.shape[0]
    depth = _depths(parent)
    demand = zipf_leaf_demand(parent, m, zipf_s, total, rng)
    w = depth_linear_recompute(depth, h10)
    if name == "tiny":
        f = requester_fetch(m, n, 100_700)
    elif name == "tree2k":
        f = pairwise_fetch(m, n, 1.0, 10.0, rng)
    elif name == "rag10k":
        f = pairwise_fetch(m, n, 1.5, 25.0, rng)
    else:
        f = pairwise_fetch(m, n, 1.0, 25.0, rng)
    return Instance(name=name, parent=parent, demand=demand, recompute_cost=w,
                    fetch_cost=f, cap=np.asarray(caps, dtype=np.int32),
                    n_starts=starts, max_rounds=rounds, order_seed=idx,
                    depth=depth)


def runtime_instance(m: int, seed: int = 11) -> Instance:
    """The shape of the paper's solver-runtime measurements at n = 10,000
    (Sec. V, solver runtime: k = 128 per worker, M = 4, 8 or 16): the
    RAG-shaped tree and demand of `rag10k` (40 templates, Zipf 0.9 over the
    leaves, 10^7 requests) split over m workers with the cyclic hardware
    factors and source-dependent fetch costs over U[1.5, 25] Gb/s; the
    paper's default start set (`n_starts = 0`: every order for m <= 5, else
    8 starts) and refinement to convergence.  The same tree for every m."""
    rng = np.random.default_rng(seed)
    parent, _ = _relabel_preorder(rag_tree(10_000, 40, rng))
    n = parent.shape[0]
    depth = _depths(parent)
    rng_m = np.random.default_rng(seed * 100 + m)
    demand = zipf_leaf_demand(parent, m, 0.9, 10 ** 7, rng_m)
    w = depth_linear_recompute(depth, H10_CYCLE[np.arange(m) % 3])
    f = pairwise_fetch(m, n, 1.5, 25.0, rng_m)
    return Instance(name=f"runtime10k_m{m}", parent=parent, demand=demand, recompute_cost=w,
                    fetch_cost=f, cap=np.full(m, 128, dtype=np.int32), n_starts=0,
                    max_rounds=0, order_seed=seed, depth=depth)


# --------------------------------------------------------------------------
# Small random instances for property and parity tests
# --------------------------------------------------------------------------

def random_forest(n: int, rng: np.random.Generator, p_root: float = 0.15,
                  shuffle: bool = True) -> np.ndarray:
    """A random forest on n nodes.  With `shuffle`, ids are permuted so the
    labels are NOT in preorder (exercises the canonical relabelling)."""
    par = np.full(n, -1, dtype=np.int32)
    for v in range(1, n):
        if rng.random() >= p_root:
            par[v] = int(rng.integers(0, v))
    if not shuffle:
        return par
    perm = rng.permutation(n)  # new label of old node v is perm[v]
    out = np.full(n, -1, dtype=np.int32)
    for v in range(n):
        if par[v] >= 0:
            out[perm[v]] = perm[par[v]]
    return out


def caterpillar(depth: int) -> np.ndarray:
    """Spine 0..depth-1 and one leaf per spine node (ids depth..2 depth-1);
    the spine child has the smaller id, so in canonical preorder every
    leaf follows the rest of the spine below its node (depth - 1 subtree
    boundaries pending at once in the DP sweep)."""
    return np.array([-1] + list(range(0, depth - 1)) + list(range(0, depth)),
                    dtype=np.int32)


def regenerated_conversation(n: int, rng: np.random.Generator) -> np.ndarray:
    """A long multi-turn conversation (a chain of n // 2 turns) whose turns
    were regenerated: the other nodes hang off uniformly random turns, one
    at a time or as short chains of their own (each next node continues the
    previous branch with probability 1/2).  Branch ids are larger than the
    chain's, so a branch follows the rest of the conversation in preorder
    and hundreds of subtree boundaries are pending at once."""
    chain = n // 2
    parent = [-1] + list(range(0, chain - 1))
    for v in range(chain, n):
        if v > chain and rng.random() < 0.5:
            parent.append(v - 1)
        else:
            parent.append(int(rng.integers(0, chain)))
    return np.array(parent, dtype=np.int32)


def random_instance(n: int, m: int, rng: np.random.Generator, *,
                    kmax: int | None = None, source_dependent: bool = True,
                    value_range: int = 50, zero_frac: float = 0.2,
                    shuffle: bool = True, parent: np.ndarray | None = None) -> Instance:
    """Small random planner input with many ties (small integer ranges), on
    a random forest or on the given tree."""
    if parent is None:
        parent = random_forest(n, rng, shuffle=shuffle)
    else:
        parent = np.asarray(parent, dtype=np.int32)
        n = parent.shape[0]
    demand = rng.integers(0, value_range, size=(m, n)).astype(np.int64)
    demand[rng.random((m, n)) < zero_frac] = 0
    w = rng.integers(0, value_range, size=(m, n)).astype(np.int64)
    if source_dependent:
        f = rng.integers(0, value_range, size=(m, m, n)).astype(np.int64)
    else:
        fr = rng.integers(0, value_range, size=(m, n)).astype(np.int64)
        f = np.broadcast_to(fr[None, :, :], (m, m, n)).copy()
    for i in range(m):
        f[i, i, :] = 0
    kmax = n + 1 if kmax is None else kmax
    cap = rng.integers(0, kmax + 1, size=m).astype(np.int32)
    depth = np.zeros(n, dtype=np.int32)
    return Instance(name="random", parent=parent, demand=demand,
                    recompute_cost=w, fetch_cost=f, cap=cap, n_starts=1,
                    max_rounds=0, order_seed=0, depth=depth)
