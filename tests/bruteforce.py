"""Independent pure-Python references used to pin the oracle on tiny inputs.

Nothing here calls the oracle or the HIP path.  Each function is written from
a definition in the paper, by enumeration rather than by the oracle's
recurrences: parent-closed sets are enumerated directly (Sec. III-A), the
objective of the requester-side model is evaluated through the
modular-plus-coverage form (Eqs. 2-4, Lemma 1), and joint optima are found
by exhaustive search over every worker's feasible sets.
"""

from __future__ import annotations

import itertools

import numpy as np


def canonical_preorder(parent) -> list[int]:
    """Roots in increasing id, children in increasing id, depth first."""
    n = len(parent)
    kids = {v: [] for v in range(-1, n)}
    for v in range(n):
        kids[int(parent[v])].append(v)
    out: list[int] = []
    # depth first with an explicit stack (trees can be thousands deep):
    # children pushed in decreasing id are popped in increasing id
    stack = sorted(kids[-1], reverse=True)
    while stack:
        v = stack.pop()
        out.append(v)
        stack.extend(sorted(kids[v], reverse=True))
    return out


def closed_sets(parent, kmax: int):
    """All parent-closed subsets with at most kmax nodes, as bool arrays."""
    n = len(parent)
    res = []
    for mask in range(1 << n):
        cnt = bin(mask).count("1")
        if cnt > kmax:
            continue
        ok = True
        for v in range(n):
            if mask >> v & 1:
                p = int(parent[v])
                if p >= 0 and not (mask >> p & 1):
                    ok = False
                    break
        if ok:
            res.append(np.array([(mask >> v) & 1 for v in range(n)], dtype=bool))
    return res


def best_closed_set(parent, profit, k):
    """Exhaustive maximum-profit parent-closed set of size <= k.  Among the
    optimal sets, returns the one whose 0/1 vector read in canonical preorder
    is lexicographically smallest."""
    order = canonical_preorder(parent)
    best_val, best_key, best_set = None, None, None
    for s in closed_sets(parent, k):
        val = int(np.sum(np.asarray(profit, dtype=object)[s])) if s.any() else 0
        key = tuple(int(s[v]) for v in order)
        if best_val is None or val > best_val or (val == best_val and key < best_key):
            best_val, best_key, best_set = val, key, s
    return best_set.astype(np.uint8), best_val


def requester_side_objective(demand, w, f_req, target) -> int:
    """F(T) of Lemma 1 (Eq. 4) for requester-side fetch costs f_m(b):
    sum_m sum_{b in T_m} a_m(b) + sum_{b in U T_m} Delta(b), with
    a_m(b) = Lambda_m(b) min{w_m(b), f_m(b)} (Eq. 2) and
    Delta(b) = sum_m Lambda_m(b) [w_m(b) - f_m(b)]_+ (Eq. 3)."""
    lam = np.asarray(demand, dtype=object)
    w = np.asarray(w, dtype=object)
    f = np.asarray(f_req, dtype=object)
    m, n = lam.shape
    total = 0
    for b in range(n):
        delta = sum(lam[r, b] * max(w[r, b] - f[r, b], 0) for r in range(m))
        covered = False
        for h in range(m):
            if target[h][b]:
                covered = True
                total += lam[h, b] * min(w[h, b], f[h, b])
        if covered:
            total += delta
    return int(total)


def requester_side_marginal(demand, w, f_req, target, h) -> list[int]:
    """Eq. (10): p_h^U(b) = a_h(b) + 1{b not in U} Delta(b), U = union of
    the other workers' sets."""
    lam = np.asarray(demand, dtype=object)
    w = np.asarray(w, dtype=object)
    f = np.asarray(f_req, dtype=object)
    m, n = lam.shape
    out = []
    for b in range(n):
        a = lam[h, b] * min(w[h, b], f[h, b])
        delta = sum(lam[r, b] * max(w[r, b] - f[r, b], 0) for r in range(m))
        in_u = any(target[l][b] for l in range(m) if l != h)
        out.append(int(a + (0 if in_u else delta)))
    return out


def pair_savings(w, f):
    """q[h][m][b] of Eq. (5), built elementwise from its case split."""
    w = np.asarray(w, dtype=np.int64)
    f = np.asarray(f, dtype=np.int64)
    m, n = w.shape
    q = np.zeros((m, m, n), dtype=np.int64)
    for h in range(m):
        for r in range(m):
            q[h, r] = w[r] if h == r else np.maximum(w[r] - f[h, r], 0)
    return q


def joint_optimum(parent, demand, w, f, cap) -> int:
    """Exhaustive OPT of problem (8) with F_pair: every combination of the
    workers' feasible parent-closed sets (tiny n and M only)."""
    lam = np.asarray(demand, dtype=np.int64)
    m, n = lam.shape
    q = pair_savings(w, f)
    sets = [np.array(closed_sets(parent, int(cap[h]))) for h in range(m)]
    best = 0
    for combo in itertools.product(*[range(len(s)) for s in sets]):
        hold = np.stack([sets[h][combo[h]] for h in range(m)])  # [m][n]
        # best saving per (requester, chunk) over holders; empty max = 0
        val = np.max(np.where(hold[:, None, :], q, 0), axis=0)
        best = max(best, int(np.sum(lam * val)))
    return best
