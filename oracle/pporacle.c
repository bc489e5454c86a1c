/*
 * pporacle.c -- plain CPU oracle of the PrefixPlace planner hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the tests, the package's smoke check and the bench's
 * CPU-baseline leg use it.  It shares no code, header, table or helper with
 * the HIP implementation.
 *
 * Everything here is the plain definition from the paper, in int64, with no
 * blocking, fusion or incremental state:
 *   - savings q_{m<-h}(b)                           Eq. (5), Sec. III-C
 *   - objective F_pair(T), max over the empty set 0  Eq. (6), Sec. III-C
 *   - worker marginal p_h(b) and v_m^{(-h)}(b)       Eq. (7), Proposition 1
 *   - rooted-tree DP D[i,j] and its backtrack        Eq. (9), Theorem 1, Algorithm 1 (RootedDP)
 *   - WorkerGreedy, coordinate refinement,
 *     order-diverse starts, best-candidate return   Sec. IV-B/IV-C, Theorem 3, Algorithm 1 (PrefixPlace)
 *   - comparator safeguards for requester-side
 *     costs (Independent, Popularity, LocalDedup)   Sec. IV-C, Algorithm 1; Sec. V-A (comparators)
 *   - epoch re-planning: switch to a fresh plan when
 *     its gain over the horizon pays for copying in
 *     the chunks it newly assigns                   Sec. IV-D; Sec. V-A (break-even requests)
 *   - the same planner on real-valued costs with the
 *     refinement tolerance epsilon                  Sec. IV-C, Algorithm 1 (REQUIRE: tolerance)
 *
 * Readings of points the paper leaves open (numbered as in the design notes):
 *   R1  DP ties: take b_i only if strictly better; skip wins ties.
 *   R2  preorder: roots, then children, in increasing node id.
 *   R3  parent = -1 attaches to the no-cost dummy root; forests allowed.
 *   R4  integer costs, so the refinement tolerance is 0 (strictly greater).
 *   R5  the greedy pass adopts every DP result.
 *   R6  standalone score of worker h = RootedDP value of p_h against the
 *       empty placement; order 0 sorts by (score desc, worker id asc).
 *   R7  order 1 = reverse of order 0; orders >= 2 are Fisher-Yates shuffles
 *       driven by SplitMix64 seeded with order_seed + start index.
 *   R8  n_starts > 0 overrides the paper's default start set; n_starts = 0
 *       selects it (M <= 5: all M! orders, lexicographic; else 8 starts).
 *   R9  max_rounds counts refinement sweeps including the last
 *       non-improving one; 0 = until a sweep accepts nothing.
 *   R10 ties between starts go to the earliest start.
 *   R11 fetch_cost[h][h][*] is ignored (q_{h<-h} = w_h).
 *   R13 capacity above n is capped to n.
 *   R18 the safeguard candidates are added only for requester-side inputs:
 *       fetch_cost[src][dst][b] equal over every src != dst (M = 1 counts
 *       as requester-side); f_m(b) is that common value.
 *   R19 Independent: RootedDP per worker with p = Lambda_m * w_m;
 *       Popularity: p = Lambda_m; LocalDedup: workers in increasing id, each
 *       RootedDP with p = a_m + 1{b not in U} Lambda_m [w_m - f_m]_+, U the
 *       union of the earlier workers' sets (the requester's own saving only,
 *       no coverage value for other requesters); capacity k_m throughout.
 *   R20 a candidate replaces the best start only if strictly better; among
 *       candidates the order Independent, Popularity, LocalDedup breaks ties.
 *   R21 one-time cost of the newly assigned chunks: sum over (m, b) with b
 *       in T'_m but not in T_m of c_m(b) = min(w_m(b), min over workers h !=
 *       m holding b in the incumbent T of f_{m<-h}(b)), under the refreshed
 *       costs.
 *   R22 the horizon H counts epochs; the re-optimized plan T' is adopted
 *       iff H * (G(T') - G(T)) > that cost (exact 128-bit comparison), G
 *       evaluated under the refreshed inputs.
 *   R24 real-valued costs (the _f64 entry points): IEEE double arithmetic,
 *       each product Lambda * x rounded before it is added (no fused
 *       multiply-add); p_h(b) sums its requester terms in increasing m; the
 *       DP takes b_i only if t > s; the comparator candidates use R18-R20
 *       with value equality of doubles.
 *   R26 G(T) on real-valued costs is the exact sum of its rounded terms
 *       Lambda_m(b) * max(...) (a sum of doubles has one exact value, while
 *       a floating-point sum depends on its order, which the paper does not
 *       fix): a refinement replacement is accepted iff the exact
 *       G(T_-h, T'_h) exceeds the exact G(T) + epsilon, both evaluated from
 *       scratch; starts and comparator candidates compare exact values
 *       (earliest on equal values); a reported objective is the exact value
 *       rounded to the nearest double (ties to even).  Re-planning rounds
 *       the exact G(T') - G(T) and the exact one-time cost to doubles and
 *       decides horizon * (G(T') - G(T)) > cost on those doubles.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <pthread.h>

enum {
    PPO_OK = 0,
    PPO_E_ARG = -1,
    PPO_E_TREE = -2,
    PPO_E_RANGE = -3,
    PPO_E_OVERFLOW = -4,
    PPO_E_NOMEM = -5
};

enum { PPO_F_NO_REFINE = 2u, PPO_F_SAFEGUARDS = 8u };

static int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }

/* ---------------------------------------------------------------- tree -- */

/* Canonical preorder (R2, R3).  order[i] = node at 0-based position i;
 * nextpos[i] = first position after the subtree of order[i] (Sec. IV-A:
 * next(i), here 0-based).  Returns PPO_E_TREE if a parent is out of range,
 * a node is its own parent, or some node never reaches a root (a cycle). */
static int preorder(int32_t n, const int32_t *parent, int32_t *order,
                    int32_t *nextpos)
{
    for (int32_t v = 0; v < n; v++) {
        if (parent[v] < -1 || parent[v] >= n || parent[v] == v)
            return PPO_E_TREE;
    }
    /* children lists, in increasing id because v is scanned upward */
    int32_t *nchild = calloc((size_t)n + 1, sizeof(int32_t));
    int32_t *start = malloc(((size_t)n + 1) * sizeof(int32_t));
    int32_t *kids = malloc((size_t)n * sizeof(int32_t));
    int32_t *fill = malloc(((size_t)n + 1) * sizeof(int32_t));
    int32_t *stack = malloc((size_t)n * sizeof(int32_t));
    int32_t *posof = malloc((size_t)n * sizeof(int32_t));
    if (!nchild || !start || !kids || !fill || !stack || !posof) {
        free(nchild); free(start); free(kids); free(fill); free(stack); free(posof);
        return PPO_E_NOMEM;
    }
    /* slot n collects the roots (children of the dummy root) */
    for (int32_t v = 0; v < n; v++)
        nchild[parent[v] < 0 ? n : parent[v]]++;
    start[0] = 0;
    for (int32_t u = 0; u < n; u++)
        start[u + 1] = start[u] + nchild[u];
    /* roots occupy [start[n], start[n] + nchild[n]) */
    for (int32_t u = 0; u <= n; u++)
        fill[u] = start[u];
    for (int32_t v = 0; v < n; v++) {
        int32_t u = parent[v] < 0 ? n : parent[v];
        kids[fill[u]++] = v;
    }
    int32_t top = 0, pos = 0;
    for (int32_t r = nchild[n] - 1; r >= 0; r--)
        stack[top++] = kids[start[n] + r];
    while (top > 0) {
        int32_t v = stack[--top];
        posof[v] = pos;
        order[pos++] = v;
        for (int32_t c = nchild[v] - 1; c >= 0; c--)
            stack[top++] = kids[start[v] + c];
    }
    int rc = PPO_OK;
    if (pos != n) {
        rc = PPO_E_TREE; /* nodes on a cycle are never reached from a root */
    } else {
        /* subtree sizes, accumulated in reverse preorder */
        int32_t *size = stack; /* reuse */
        for (int32_t i = 0; i < n; i++)
            size[i] = 1;
        for (int32_t i = n - 1; i >= 0; i--) {
            int32_t v = order[i];
            if (parent[v] >= 0)
                size[posof[parent[v]]] += size[i];
        }
        for (int32_t i = 0; i < n; i++)
            nextpos[i] = i + size[i];
    }
    free(nchild); free(start); free(kids); free(fill); free(stack); free(posof);
    return rc;
}

/* ----------------------------------------------------------- RootedDP -- */

/* Eq. (9) with 1-based preorder positions i = 1..n, nxt(i) = next(i):
 *   D[i][j] = max(D[next(i)][j], p(b_i) + D[i+1][j-1]),
 *   D[n+1][j] = 0, D[i][0] = 0.
 * The whole (n+2) x (k'+1) table is kept (Theorem 1: O(nk) memory), and the
 * backtrack compares table values (R1: take only if strictly better).
 * profit_pos[i-1] is p(b_i); sel_pos[i-1] is set to 1 for chosen b_i. */
static int rooted_dp_pos(int32_t n, const int32_t *nextpos,
                         const int64_t *profit_pos, int32_t k,
                         uint8_t *sel_pos, int64_t *value)
{
    int64_t kk = k < n ? k : n; /* R13 */
    memset(sel_pos, 0, (size_t)n);
    if (kk <= 0) {
        *value = 0;
        return PPO_OK;
    }
    size_t W = (size_t)kk + 1;
    int64_t *D = calloc(((size_t)n + 2) * W, sizeof(int64_t));
    if (!D)
        return PPO_E_NOMEM;
#define CELL(i, j) D[(size_t)(i) * W + (size_t)(j)]
    for (int64_t i = n; i >= 1; i--) {
        int64_t nx = (int64_t)nextpos[i - 1] + 1; /* 1-based next(i) */
        int64_t p = profit_pos[i - 1];
        for (int64_t j = 1; j <= kk; j++) {
            int64_t s = CELL(nx, j);          /* skip b_i and its subtree */
            int64_t t = p + CELL(i + 1, j - 1); /* take b_i */
            CELL(i, j) = max64(s, t);
        }
    }
    *value = CELL(1, kk);
    int64_t i = 1, j = kk;
    while (i <= n && j > 0) {
        int64_t nx = (int64_t)nextpos[i - 1] + 1;
        int64_t s = CELL(nx, j);
        int64_t t = profit_pos[i - 1] + CELL(i + 1, j - 1);
        if (t > s) {
            sel_pos[i - 1] = 1;
            i += 1;
            j -= 1;
        } else {
            i = nx;
        }
    }
#undef CELL
    free(D);
    return PPO_OK;
}

/* ------------------------------------------------------------ savings -- */

/* Eq. (5): q_{m<-h}(b) = w_m(b) if h == m, else [w_m(b) - f_{m<-h}(b)]_+.
 * fetch is laid out [src=h][dst=m][b]. */
static int64_t q_save(int32_t n, int32_t m, const int64_t *w, const int64_t *f,
                      int32_t h, int32_t req, int32_t b)
{
    int64_t wm = w[(size_t)req * n + b];
    if (h == req)
        return wm;
    int64_t fh = f[((size_t)h * m + req) * n + b];
    return max64(wm - fh, 0);
}

/* Eq. (6): G(T) = sum_b sum_m Lambda_m(b) * max({q_{m<-h}(b) : b in T_h} u {0}). */
static int64_t objective_full(int32_t n, int32_t m, const int64_t *lam,
                              const int64_t *w, const int64_t *f,
                              const uint8_t *tgt)
{
    int64_t g = 0;
    for (int32_t b = 0; b < n; b++) {
        for (int32_t r = 0; r < m; r++) {
            int64_t best = 0;
            for (int32_t h = 0; h < m; h++)
                if (tgt[(size_t)h * n + b])
                    best = max64(best, q_save(n, m, w, f, h, r, b));
            g += lam[(size_t)r * n + b] * best;
        }
    }
    return g;
}

/* Eq. (7) / Proposition 1: with every worker but h fixed,
 *   v_m(b) = max({q_{m<-l}(b) : l != h, b in T_l} u {0}),
 *   p_h(b) = sum_m Lambda_m(b) [q_{m<-h}(b) - v_m(b)]_+,
 * and G(T_{-h}) = sum_{m,b} Lambda_m(b) v_m(b). */
static void marginal_full(int32_t n, int32_t m, const int64_t *lam,
                          const int64_t *w, const int64_t *f,
                          const uint8_t *tgt, int32_t h, int64_t *profit,
                          int64_t *g_without)
{
    int64_t g = 0;
    for (int32_t b = 0; b < n; b++) {
        int64_t p = 0;
        for (int32_t r = 0; r < m; r++) {
            int64_t v = 0;
            for (int32_t l = 0; l < m; l++)
                if (l != h && tgt[(size_t)l * n + b])
                    v = max64(v, q_save(n, m, w, f, l, r, b));
            int64_t L = lam[(size_t)r * n + b];
            p += L * max64(q_save(n, m, w, f, h, r, b) - v, 0);
            g += L * v;
        }
        profit[b] = p;
    }
    if (g_without)
        *g_without = g;
}

/* --------------------------------------------------------- validation -- */

static int validate(int32_t n, int32_t m, const int32_t *parent,
                    const int64_t *lam, const int64_t *w, const int64_t *f,
                    const int32_t *cap)
{
    if (n < 1 || m < 1 || m > 255 || !parent || !lam || !w || !f || !cap)
        return PPO_E_ARG;
    for (int32_t v = 0; v < n; v++)
        if (parent[v] < -1 || parent[v] >= n || parent[v] == v)
            return PPO_E_TREE;
    size_t mn = (size_t)m * n;
    for (size_t x = 0; x < mn; x++)
        if (lam[x] < 0 || w[x] < 0)
            return PPO_E_RANGE;
    for (size_t x = 0; x < mn * (size_t)m; x++)
        if (f[x] < 0)
            return PPO_E_RANGE;
    for (int32_t r = 0; r < m; r++)
        if (cap[r] < 0)
            return PPO_E_RANGE;
    /* every p, D and G value is at most sum Lambda * w; it must fit int64 */
    unsigned __int128 tot = 0;
    for (size_t x = 0; x < mn; x++) {
        tot += (unsigned __int128)(uint64_t)lam[x] * (uint64_t)w[x];
        if (tot > (unsigned __int128)INT64_MAX)
            return PPO_E_OVERFLOW;
    }
    return PPO_OK;
}

/* Value checks shared by the entry points that take no tree. */
static int validate_values(int32_t n, int32_t m, const int64_t *lam,
                           const int64_t *w, const int64_t *f)
{
    size_t mn = (size_t)m * n;
    for (size_t x = 0; x < mn; x++)
        if (lam[x] < 0 || w[x] < 0)
            return PPO_E_RANGE;
    for (size_t x = 0; x < mn * (size_t)m; x++)
        if (f[x] < 0)
            return PPO_E_RANGE;
    unsigned __int128 tot = 0;
    for (size_t x = 0; x < mn; x++) {
        tot += (unsigned __int128)(uint64_t)lam[x] * (uint64_t)w[x];
        if (tot > (unsigned __int128)INT64_MAX)
            return PPO_E_OVERFLOW;
    }
    return PPO_OK;
}

/* ------------------------------------------------------------- orders -- */

/* SplitMix64 (Steele, Lea & Flood, OOPSLA 2014), in the published form. */
static uint64_t splitmix64(uint64_t *x)
{
    uint64_t z = (*x += 0x9e3779b97f4a7c15ULL);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

/* Lexicographic successor of a permutation; returns 0 after the last one. */
static int next_perm(int32_t *a, int32_t m)
{
    int32_t i = m - 2;
    while (i >= 0 && a[i] >= a[i + 1])
        i--;
    if (i < 0)
        return 0;
    int32_t j = m - 1;
    while (a[j] <= a[i])
        j--;
    int32_t t = a[i]; a[i] = a[j]; a[j] = t;
    for (int32_t l = i + 1, r = m - 1; l < r; l++, r--) {
        t = a[l]; a[l] = a[r]; a[r] = t;
    }
    return 1;
}

static int64_t factorial(int32_t m)
{
    int64_t f = 1;
    for (int32_t i = 2; i <= m; i++)
        f *= i;
    return f;
}

/* Number of starts the options select (R8). */
int32_t ppo_num_starts(int32_t m, int32_t n_starts)
{
    if (n_starts > 0)
        return n_starts;
    if (m <= 5)
        return (int32_t)factorial(m);
    return 8;
}

/* Start orders (Sec. IV-C; R6-R8).  standalone[h] is worker h's score. */
int ppo_orders(int32_t m, int32_t n_starts, uint64_t order_seed,
               const int64_t *standalone, int32_t *orders)
{
    if (m < 1 || m > 255 || n_starts < 0 || !standalone || !orders)
        return PPO_E_ARG;
    int32_t S = ppo_num_starts(m, n_starts);
    if (n_starts == 0 && m <= 5) {
        int32_t *a = orders;
        for (int32_t h = 0; h < m; h++)
            a[h] = h;
        for (int32_t s = 1; s < S; s++) {
            memcpy(orders + (size_t)s * m, orders + (size_t)(s - 1) * m,
                   (size_t)m * sizeof(int32_t));
            next_perm(orders + (size_t)s * m, m);
        }
        return PPO_OK;
    }
    /* order 0: score descending, then id ascending (selection sort) */
    int32_t *o0 = orders;
    for (int32_t h = 0; h < m; h++)
        o0[h] = h;
    for (int32_t a = 0; a < m; a++) {
        int32_t best = a;
        for (int32_t c = a + 1; c < m; c++) {
            int64_t sc = standalone[o0[c]], sb = standalone[o0[best]];
            if (sc > sb || (sc == sb && o0[c] < o0[best]))
                best = c;
        }
        int32_t t = o0[a]; o0[a] = o0[best]; o0[best] = t;
    }
    for (int32_t s = 1; s < S; s++) {
        int32_t *o = orders + (size_t)s * m;
        if (s == 1) {
            for (int32_t h = 0; h < m; h++)
                o[h] = o0[m - 1 - h];
        } else {
            uint64_t x = order_seed + (uint64_t)s;
            for (int32_t h = 0; h < m; h++)
                o[h] = h;
            for (int32_t i = m - 1; i >= 1; i--) {
                int32_t j = (int32_t)(splitmix64(&x) % (uint64_t)(i + 1));
                int32_t t = o[i]; o[i] = o[j]; o[j] = t;
            }
        }
    }
    return PPO_OK;
}

/* Raw SplitMix64 stream, exported so tests can pin it to published values. */
void ppo_splitmix64_stream(uint64_t seed, int32_t count, uint64_t *out)
{
    uint64_t x = seed;
    for (int32_t i = 0; i < count; i++)
        out[i] = splitmix64(&x);
}

/* ----------------------------------------------------- per-kernel ABI -- */

int ppo_preorder(int32_t n, const int32_t *parent, int32_t *order,
                 int32_t *nextpos)
{
    if (n < 1 || !parent || !order || !nextpos)
        return PPO_E_ARG;
    return preorder(n, parent, order, nextpos);
}

/* One exact rooted-tree solve in caller ids (Theorem 1). */
int ppo_rooted_dp(int32_t n, const int32_t *parent, const int64_t *profit,
                  int32_t k, uint8_t *selected, int64_t *value)
{
    if (n < 1 || !parent || !profit || !selected || !value || k < 0)
        return PPO_E_ARG;
    for (int32_t b = 0; b < n; b++)
        if (profit[b] < 0)
            return PPO_E_RANGE;
    int32_t *order = malloc((size_t)n * sizeof(int32_t));
    int32_t *nextpos = malloc((size_t)n * sizeof(int32_t));
    int64_t *pp = malloc((size_t)n * sizeof(int64_t));
    uint8_t *sp = malloc((size_t)n);
    int rc = PPO_E_NOMEM;
    if (order && nextpos && pp && sp) {
        rc = preorder(n, parent, order, nextpos);
        if (rc == PPO_OK) {
            /* sum of profits must fit int64 */
            unsigned __int128 tot = 0;
            for (int32_t b = 0; b < n; b++)
                tot += (uint64_t)profit[b];
            if (tot > (unsigned __int128)INT64_MAX)
                rc = PPO_E_OVERFLOW;
        }
        if (rc == PPO_OK) {
            for (int32_t i = 0; i < n; i++)
                pp[i] = profit[order[i]];
            int64_t val = 0;
            rc = rooted_dp_pos(n, nextpos, pp, k, sp, &val);
            if (rc == PPO_OK) {
                for (int32_t i = 0; i < n; i++)
                    selected[order[i]] = sp[i];
                *value = val;
            }
        }
    }
    free(order); free(nextpos); free(pp); free(sp);
    return rc;
}

int ppo_marginal(int32_t n, int32_t m, const int64_t *demand,
                 const int64_t *recompute_cost, const int64_t *fetch_cost,
                 const uint8_t *target, int32_t h, int64_t *profit,
                 int64_t *g_without_h)
{
    if (n < 1 || m < 1 || m > 255 || !demand || !recompute_cost ||
        !fetch_cost || !target || !profit || h < 0 || h >= m)
        return PPO_E_ARG;
    int rc = validate_values(n, m, demand, recompute_cost, fetch_cost);
    if (rc != PPO_OK)
        return rc;
    marginal_full(n, m, demand, recompute_cost, fetch_cost, target, h, profit,
                  g_without_h);
    return PPO_OK;
}

int ppo_objective(int32_t n, int32_t m, const int64_t *demand,
                  const int64_t *recompute_cost, const int64_t *fetch_cost,
                  const uint8_t *target, int64_t *objective)
{
    if (n < 1 || m < 1 || m > 255 || !demand || !recompute_cost ||
        !fetch_cost || !target || !objective)
        return PPO_E_ARG;
    int rc = validate_values(n, m, demand, recompute_cost, fetch_cost);
    if (rc != PPO_OK)
        return rc;
    *objective = objective_full(n, m, demand, recompute_cost, fetch_cost,
                                target);
    return PPO_OK;
}

/* ---------------------------------------------------------- safeguards -- */

/* R18: 1 when fetch_cost[src][dst][b] is the same for every src != dst. */
int ppo_requester_side(int32_t n, int32_t m, const int64_t *fetch_cost)
{
    for (int32_t dst = 0; dst < m; dst++) {
        int32_t first = dst == 0 ? 1 : 0;
        for (int32_t src = first + 1; src < m; src++) {
            if (src == dst)
                continue;
            for (int32_t b = 0; b < n; b++)
                if (fetch_cost[((size_t)src * m + dst) * n + b] !=
                    fetch_cost[((size_t)first * m + dst) * n + b])
                    return 0;
        }
    }
    return 1;
}

/* The three comparator placements of Sec. IV-C (R19), each a RootedDP per
 * worker, and their objective F (= F_pair for requester-side inputs).
 *   targets [3][m][n] out (caller ids): Independent, Popularity, LocalDedup
 *   objs    [3] out */
int ppo_candidates(int32_t n, int32_t m, const int32_t *parent,
                   const int64_t *demand, const int64_t *recompute_cost,
                   const int64_t *fetch_cost, const int32_t *cap,
                   uint8_t *targets, int64_t *objs)
{
    int rc = validate(n, m, parent, demand, recompute_cost, fetch_cost, cap);
    if (rc != PPO_OK)
        return rc;
    if (!targets || !objs)
        return PPO_E_ARG;
    int32_t *order = malloc((size_t)n * sizeof(int32_t));
    int32_t *nextpos = malloc((size_t)n * sizeof(int32_t));
    int64_t *pp = malloc((size_t)n * sizeof(int64_t));
    uint8_t *sp = malloc((size_t)n);
    rc = PPO_E_NOMEM;
    if (!order || !nextpos || !pp || !sp)
        goto out;
    rc = preorder(n, parent, order, nextpos);
    if (rc != PPO_OK)
        goto out;
    memset(targets, 0, (size_t)3 * m * n);
    for (int32_t c = 0; c < 3; c++) {
        uint8_t *tg = targets + (size_t)c * m * n;
        for (int32_t h = 0; h < m; h++) {
            const int64_t *lam = demand + (size_t)h * n;
            const int64_t *w = recompute_cost + (size_t)h * n;
            /* f_h(b): the common off-diagonal fetch cost (R18) */
            int32_t src = h == 0 ? 1 : 0;
            const int64_t *f = m > 1 ? fetch_cost + ((size_t)src * m + h) * n : NULL;
            for (int32_t i = 0; i < n; i++) {
                int32_t b = order[i];
                int64_t p;
                if (c == 0) {
                    p = lam[b] * w[b];                  /* Independent */
                } else if (c == 1) {
                    p = lam[b];                         /* Popularity */
                } else if (!f) {
                    p = lam[b] * w[b];                  /* LocalDedup, M = 1 */
                } else {
                    int covered = 0;                    /* b in U (earlier ids) */
                    for (int32_t l = 0; l < h; l++)
                        covered |= tg[(size_t)l * n + b];
                    int64_t a = lam[b] * (w[b] < f[b] ? w[b] : f[b]);
                    int64_t own = lam[b] * max64(w[b] - f[b], 0);
                    p = covered ? a : a + own;          /* LocalDedup */
                }
                pp[i] = p;
            }
            int64_t v;
            rc = rooted_dp_pos(n, nextpos, pp, cap[h], sp, &v);
            if (rc != PPO_OK)
                goto out;
            for (int32_t i = 0; i < n; i++)
                tg[(size_t)h * n + order[i]] = sp[i];
        }
        objs[c] = objective_full(n, m, demand, recompute_cost, fetch_cost, tg);
    }
    rc = PPO_OK;
out:
    free(order); free(nextpos); free(pp); free(sp);
    return rc;
}

/* ------------------------------------------------------------ re-plan -- */

int ppo_plan(int32_t n, int32_t m, const int32_t *parent, const int64_t *demand,
             const int64_t *recompute_cost, const int64_t *fetch_cost,
             const int32_t *cap, int32_t n_starts, int32_t max_rounds,
             uint64_t order_seed, const int32_t *orders_in, uint32_t flags,
             int32_t threads, uint8_t *target, int64_t *objective,
             int64_t *standalone_out, int32_t *orders_out,
             int64_t *start_objective, int32_t *start_sweeps,
             int32_t *start_accepts, int64_t *info, int64_t *safeguard_obj);

/* R21: one-time cost of materializing the chunks of `proposal` that the
 * incumbent does not place at the same worker (both [m][n], caller ids). */
static unsigned __int128 materialization_cost(int32_t n, int32_t m,
                                              const int64_t *w,
                                              const int64_t *f,
                                              const uint8_t *incumbent,
                                              const uint8_t *proposal)
{
    unsigned __int128 total = 0;
    for (int32_t r = 0; r < m; r++)
        for (int32_t b = 0; b < n; b++) {
            if (!proposal[(size_t)r * n + b] || incumbent[(size_t)r * n + b])
                continue;
            int64_t c = w[(size_t)r * n + b];  /* recompute */
            for (int32_t h = 0; h < m; h++)     /* or fetch from a holder */
                if (h != r && incumbent[(size_t)h * n + b]) {
                    int64_t fh = f[((size_t)h * m + r) * n + b];
                    if (fh < c)
                        c = fh;
                }
            total += (uint64_t)c;
        }
    return total;
}

int ppo_materialization_cost(int32_t n, int32_t m, const int64_t *recompute_cost,
                             const int64_t *fetch_cost, const uint8_t *incumbent,
                             const uint8_t *proposal, int64_t *cost)
{
    if (n < 1 || m < 1 || !recompute_cost || !fetch_cost || !incumbent ||
        !proposal || !cost)
        return PPO_E_ARG;
    unsigned __int128 c = materialization_cost(n, m, recompute_cost, fetch_cost,
                                               incumbent, proposal);
    if (c > (unsigned __int128)INT64_MAX)
        return PPO_E_OVERFLOW;
    *cost = (int64_t)c;
    return PPO_OK;
}

/* Epoch re-planning (Sec. IV-D): plan the refreshed inputs with ppo_plan's
 * options, evaluate the incumbent under them, and adopt the new plan iff the
 * saving over `horizon` epochs exceeds the one-time materialization cost
 * (R21, R22).
 *   incumbent [m][n]   the current placement (caller ids)
 *   target    [m][n]   out: the placement to use (proposal if adopted)
 *   proposal  [m][n]   out (may be NULL): the re-optimized plan
 *   result[4]          out: adopt (0/1), G(incumbent), G(proposal), cost */
int ppo_replan(int32_t n, int32_t m, const int32_t *parent, const int64_t *demand,
               const int64_t *recompute_cost, const int64_t *fetch_cost,
               const int32_t *cap, const uint8_t *incumbent, int64_t horizon,
               int32_t n_starts, int32_t max_rounds, uint64_t order_seed,
               uint32_t flags, int32_t threads, uint8_t *target,
               uint8_t *proposal, int64_t *result)
{
    if (!incumbent || !target || !result || horizon < 0)
        return PPO_E_ARG;
    int rc = validate(n, m, parent, demand, recompute_cost, fetch_cost, cap);
    if (rc != PPO_OK)
        return rc;
    for (size_t x = 0; x < (size_t)m * n; x++)
        if (incumbent[x] > 1)
            return PPO_E_ARG;  /* a placement is a 0/1 matrix */
    uint8_t *prop = malloc((size_t)m * n);
    if (!prop)
        return PPO_E_NOMEM;
    int64_t g_new;
    rc = ppo_plan(n, m, parent, demand, recompute_cost, fetch_cost, cap,
                  n_starts, max_rounds, order_seed, NULL, flags, threads, prop,
                  &g_new, NULL, NULL, NULL, NULL, NULL, NULL, NULL);
    if (rc != PPO_OK) {
        free(prop);
        return rc;
    }
    int64_t g_inc = objective_full(n, m, demand, recompute_cost, fetch_cost,
                                   incumbent);
    unsigned __int128 cost = materialization_cost(n, m, recompute_cost,
                                                  fetch_cost, incumbent, prop);
    if (cost > (unsigned __int128)INT64_MAX) {
        free(prop);
        return PPO_E_OVERFLOW;
    }
    /* H * (G' - G) > cost; G' - G < 0 never adopts (cost >= 0) */
    int adopt = 0;
    if (g_new > g_inc) {
        unsigned __int128 gain = (unsigned __int128)(uint64_t)(g_new - g_inc) *
                                 (uint64_t)horizon;
        adopt = gain > cost;
    }
    memcpy(target, adopt ? prop : incumbent, (size_t)m * n);
    if (proposal)
        memcpy(proposal, prop, (size_t)m * n);
    result[0] = adopt;
    result[1] = g_inc;
    result[2] = g_new;
    result[3] = (int64_t)cost;
    free(prop);
    return PPO_OK;
}

/* --------------------------------------------------------------- plan -- */

typedef struct {
    int32_t n, m;
    const int64_t *lam, *w, *f;
    const int32_t *cap;
    const int32_t *order, *nextpos;
    int32_t max_rounds;
    uint32_t flags;
} plan_in;

/* one worker update: p = marginal(h, T) with T_h treated as empty, then
 * RootedDP(p, k_h); writes the chosen set into cand (caller ids). */
static int worker_update(const plan_in *in, const uint8_t *tgt, int32_t h,
                         int64_t *profit, int64_t *pp, uint8_t *sp,
                         uint8_t *cand, int64_t *dpval)
{
    int32_t n = in->n;
    marginal_full(n, in->m, in->lam, in->w, in->f, tgt, h, profit, NULL);
    for (int32_t i = 0; i < n; i++)
        pp[i] = profit[in->order[i]];
    int rc = rooted_dp_pos(n, in->nextpos, pp, in->cap[h], sp, dpval);
    if (rc != PPO_OK)
        return rc;
    for (int32_t i = 0; i < n; i++)
        cand[in->order[i]] = sp[i];
    return PPO_OK;
}

/* Algorithm 1, one start: WorkerGreedy in the fixed order, then coordinate
 * refinement sweeps that accept only strict improvements of G (R4, R5, R9). */
static int run_start(const plan_in *in, const int32_t *pi, uint8_t *tgt,
                     int64_t *obj, int32_t *sweeps, int32_t *accepts)
{
    int32_t n = in->n, m = in->m;
    int64_t *profit = malloc((size_t)n * sizeof(int64_t));
    int64_t *pp = malloc((size_t)n * sizeof(int64_t));
    uint8_t *sp = malloc((size_t)n);
    uint8_t *cand = malloc((size_t)n);
    uint8_t *old = malloc((size_t)n);
    int rc = PPO_E_NOMEM;
    if (!profit || !pp || !sp || !cand || !old)
        goto out;
    memset(tgt, 0, (size_t)m * n);
    int64_t v;
    for (int32_t a = 0; a < m; a++) {  /* greedy pass: always adopt */
        int32_t h = pi[a];
        rc = worker_update(in, tgt, h, profit, pp, sp, cand, &v);
        if (rc != PPO_OK)
            goto out;
        memcpy(tgt + (size_t)h * n, cand, (size_t)n);
    }
    int32_t r = 0, acc = 0;
    if (!(in->flags & PPO_F_NO_REFINE)) {
        int improved;
        do {
            improved = 0;
            for (int32_t a = 0; a < m; a++) {
                int32_t h = pi[a];
                int64_t g_old = objective_full(n, m, in->lam, in->w, in->f, tgt);
                uint8_t *th = tgt + (size_t)h * n;
                memcpy(old, th, (size_t)n);
                memset(th, 0, (size_t)n);
                rc = worker_update(in, tgt, h, profit, pp, sp, cand, &v);
                if (rc != PPO_OK)
                    goto out;
                memcpy(th, cand, (size_t)n);
                int64_t g_new = objective_full(n, m, in->lam, in->w, in->f, tgt);
                if (g_new > g_old) {
                    improved = 1;
                    acc++;
                } else {
                    memcpy(th, old, (size_t)n);
                }
            }
            r++;
        } while (improved && !(in->max_rounds > 0 && r == in->max_rounds));
    }
    *obj = objective_full(n, m, in->lam, in->w, in->f, tgt);
    *sweeps = r;
    *accepts = acc;
    rc = PPO_OK;
out:
    free(profit); free(pp); free(sp); free(cand); free(old);
    return rc;
}

typedef struct {
    const plan_in *in;
    int32_t S;
    const int32_t *orders;
    uint8_t *tgts;        /* [S][m][n] */
    int64_t *obj;
    int32_t *sweeps, *accepts;
    int *rcs;
    /* standalone phase */
    int64_t *standalone;
    int phase;
    int32_t next_job;
    pthread_mutex_t mu;
} plan_work;

static int32_t take_job(plan_work *pw, int32_t limit)
{
    pthread_mutex_lock(&pw->mu);
    int32_t j = pw->next_job < limit ? pw->next_job++ : -1;
    pthread_mutex_unlock(&pw->mu);
    return j;
}

static void *plan_worker(void *arg)
{
    plan_work *pw = arg;
    const plan_in *in = pw->in;
    int32_t n = in->n, m = in->m;
    if (pw->phase == 0) {
        /* R6: standalone score = DP value of p_h against the empty placement */
        uint8_t *empty = calloc((size_t)m * n, 1);
        int64_t *profit = malloc((size_t)n * sizeof(int64_t));
        int64_t *pp = malloc((size_t)n * sizeof(int64_t));
        uint8_t *sp = malloc((size_t)n);
        uint8_t *cand = malloc((size_t)n);
        int32_t h;
        while ((h = take_job(pw, m)) >= 0) {
            if (!empty || !profit || !pp || !sp || !cand) {
                pw->rcs[h] = PPO_E_NOMEM;
                continue;
            }
            pw->rcs[h] = worker_update(in, empty, h, profit, pp, sp, cand,
                                       &pw->standalone[h]);
        }
        free(empty); free(profit); free(pp); free(sp); free(cand);
    } else {
        int32_t s;
        while ((s = take_job(pw, pw->S)) >= 0)
            pw->rcs[s] = run_start(in, pw->orders + (size_t)s * m,
                                   pw->tgts + (size_t)s * m * n, &pw->obj[s],
                                   &pw->sweeps[s], &pw->accepts[s]);
    }
    return NULL;
}

static int run_phase(plan_work *pw, int phase, int32_t jobs, int32_t threads)
{
    pw->phase = phase;
    pw->next_job = 0;
    int32_t T = threads < 1 ? 1 : threads;
    if (T > jobs)
        T = jobs;
    pthread_t *tid = malloc((size_t)T * sizeof(pthread_t));
    if (!tid)
        return PPO_E_NOMEM;
    int32_t started = 0;
    for (int32_t t = 0; t < T; t++) {
        if (pthread_create(&tid[t], NULL, plan_worker, pw) != 0)
            break;
        started++;
    }
    if (started == 0)
        plan_worker(pw);
    for (int32_t t = 0; t < started; t++)
        pthread_join(tid[t], NULL);
    free(tid);
    for (int32_t j = 0; j < jobs; j++)
        if (pw->rcs[j] != PPO_OK)
            return pw->rcs[j];
    return PPO_OK;
}

/* The whole planner (Algorithm 1 with the readings above).
 *   target[m][n]          out: the returned placement, caller ids
 *   objective             out: G of the returned placement
 *   standalone_out[m]     optional out: standalone scores (R6)
 *   orders_out[S][m]      optional out: the start orders used
 *   start_objective[S], start_sweeps[S], start_accepts[S]: optional outs
 *   info[5] (int64)       optional out: index of the returned candidate
 *                         (start s, or S + c for safeguard c), executed
 *                         worker updates, executed DP cells (sum of
 *                         n * min(k_h, n) over updates), number of starts S,
 *                         1 if the safeguard candidates were evaluated.
 *   safeguard_obj[3]      optional out: their objectives (0 if not run). */
int ppo_plan(int32_t n, int32_t m, const int32_t *parent, const int64_t *demand,
             const int64_t *recompute_cost, const int64_t *fetch_cost,
             const int32_t *cap, int32_t n_starts, int32_t max_rounds,
             uint64_t order_seed, const int32_t *orders_in, uint32_t flags,
             int32_t threads, uint8_t *target, int64_t *objective,
             int64_t *standalone_out, int32_t *orders_out,
             int64_t *start_objective, int32_t *start_sweeps,
             int32_t *start_accepts, int64_t *info, int64_t *safeguard_obj)
{
    int rc = validate(n, m, parent, demand, recompute_cost, fetch_cost, cap);
    if (rc != PPO_OK)
        return rc;
    if (n_starts < 0 || max_rounds < 0 || !target || !objective)
        return PPO_E_ARG;
    int32_t S = ppo_num_starts(m, n_starts);
    if (orders_in) {
        if (n_starts < 1)
            return PPO_E_ARG;
        for (int32_t s = 0; s < S; s++) {
            /* each explicit order must be a permutation of 0..m-1 */
            uint8_t seen[256] = {0};
            for (int32_t a = 0; a < m; a++) {
                int32_t h = orders_in[(size_t)s * m + a];
                if (h < 0 || h >= m || seen[h])
                    return PPO_E_ARG;
                seen[h] = 1;
            }
        }
    }
    int32_t *order = malloc((size_t)n * sizeof(int32_t));
    int32_t *nextpos = malloc((size_t)n * sizeof(int32_t));
    int32_t *orders = malloc((size_t)S * m * sizeof(int32_t));
    int64_t *standalone = malloc((size_t)m * sizeof(int64_t));
    uint8_t *tgts = malloc((size_t)S * m * n);
    uint8_t *cands = NULL;
    int64_t *obj = malloc((size_t)S * sizeof(int64_t));
    int32_t *sw = malloc((size_t)S * sizeof(int32_t));
    int32_t *ac = malloc((size_t)S * sizeof(int32_t));
    int *rcs = malloc((size_t)(S > m ? S : m) * sizeof(int));
    rc = PPO_E_NOMEM;
    if (!order || !nextpos || !orders || !standalone || !tgts || !obj ||
        !sw || !ac || !rcs)
        goto out;
    rc = preorder(n, parent, order, nextpos);
    if (rc != PPO_OK)
        goto out;
    plan_in in = {n, m, demand, recompute_cost, fetch_cost, cap, order,
                  nextpos, max_rounds, flags};
    plan_work pw;
    memset(&pw, 0, sizeof pw);
    pw.in = &in;
    pw.S = S;
    pw.tgts = tgts;
    pw.obj = obj;
    pw.sweeps = sw;
    pw.accepts = ac;
    pw.rcs = rcs;
    pw.standalone = standalone;
    pthread_mutex_init(&pw.mu, NULL);
    rc = run_phase(&pw, 0, m, threads);
    if (rc == PPO_OK) {
        if (orders_in)
            memcpy(orders, orders_in, (size_t)S * m * sizeof(int32_t));
        else
            rc = ppo_orders(m, n_starts, order_seed, standalone, orders);
    }
    if (rc == PPO_OK) {
        pw.orders = orders;
        rc = run_phase(&pw, 1, S, threads);
    }
    pthread_mutex_destroy(&pw.mu);
    if (rc != PPO_OK)
        goto out;
    /* Algorithm 1: return the best candidate; R10: earliest start on ties */
    int32_t best = 0;
    for (int32_t s = 1; s < S; s++)
        if (obj[s] > obj[best])
            best = s;
    const uint8_t *won = tgts + (size_t)best * m * n;
    int64_t won_obj = obj[best];
    int64_t sg_obj[3] = {0, 0, 0};
    int sg_run = 0;
    if ((flags & PPO_F_SAFEGUARDS) && ppo_requester_side(n, m, fetch_cost)) {
        cands = malloc((size_t)3 * m * n);
        rc = PPO_E_NOMEM;
        if (!cands)
            goto out;
        rc = ppo_candidates(n, m, parent, demand, recompute_cost, fetch_cost,
                            cap, cands, sg_obj);
        if (rc != PPO_OK)
            goto out;
        sg_run = 1;
        for (int32_t c = 0; c < 3; c++)  /* R20 */
            if (sg_obj[c] > won_obj) {
                won_obj = sg_obj[c];
                won = cands + (size_t)c * m * n;
                best = S + c;
            }
    }
    memcpy(target, won, (size_t)m * n);
    *objective = won_obj;
    int64_t updates = m, cells = 0;
    for (int32_t h = 0; h < m; h++)
        cells += (int64_t)n * (cap[h] < n ? cap[h] : n);
    int64_t cells_per_pass = cells;
    for (int32_t s = 0; s < S; s++) {
        updates += (int64_t)m * (1 + sw[s]);
        cells += cells_per_pass * (1 + sw[s]);
    }
    if (standalone_out)
        memcpy(standalone_out, standalone, (size_t)m * sizeof(int64_t));
    if (orders_out)
        memcpy(orders_out, orders, (size_t)S * m * sizeof(int32_t));
    if (start_objective)
        memcpy(start_objective, obj, (size_t)S * sizeof(int64_t));
    if (start_sweeps)
        memcpy(start_sweeps, sw, (size_t)S * sizeof(int32_t));
    if (start_accepts)
        memcpy(start_accepts, ac, (size_t)S * sizeof(int32_t));
    if (sg_run) {  /* 3M more DP updates */
        updates += 3 * (int64_t)m;
        cells += 3 * cells_per_pass;
    }
    if (info) {
        info[0] = best;
        info[1] = updates;
        info[2] = cells;
        info[3] = S;
        info[4] = sg_run;
    }
    if (safeguard_obj)
        memcpy(safeguard_obj, sg_obj, sizeof sg_obj);
    rc = PPO_OK;
out:
    free(order); free(nextpos); free(orders); free(standalone); free(tgts);
    free(obj); free(sw); free(ac); free(rcs); free(cands);
    return rc;
}

/* ------------------------------------------------ real-valued costs -- */

/* The same definitions on IEEE doubles (R24).  Costs must be finite and
 * non-negative.  Written out separately from the integer path so that each
 * reads as its equation. */

static double maxd(double a, double b) { return a > b ? a : b; }

static int finite_nonneg(double x) { return x >= 0.0 && x <= 1.7976931348623157e308; }

static int validate_f64(int32_t n, int32_t m, const int32_t *parent,
                        const double *lam, const double *w, const double *f,
                        const int32_t *cap)
{
    if (n < 1 || m < 1 || m > 255 || !parent || !lam || !w || !f || !cap)
        return PPO_E_ARG;
    for (int32_t v = 0; v < n; v++)
        if (parent[v] < -1 || parent[v] >= n || parent[v] == v)
            return PPO_E_TREE;
    size_t mn = (size_t)m * n;
    for (size_t x = 0; x < mn; x++)
        if (!finite_nonneg(lam[x]) || !finite_nonneg(w[x]))
            return PPO_E_RANGE;
    for (size_t x = 0; x < mn * (size_t)m; x++)
        if (!finite_nonneg(f[x]))
            return PPO_E_RANGE;
    for (int32_t r = 0; r < m; r++)
        if (cap[r] < 0)
            return PPO_E_RANGE;
    return PPO_OK;
}

/* Eq. (5) */
static double q_save_f64(int32_t n, int32_t m, const double *w, const double *f,
                         int32_t h, int32_t req, int32_t b)
{
    double wm = w[(size_t)req * n + b];
    if (h == req)
        return wm;
    double d = wm - f[((size_t)h * m + req) * n + b];
    return maxd(d, 0.0);
}

/* Exact sums of non-negative doubles (R26).  Every finite double x >= 0 is
 * an integer multiple of 2^-1074, so a sum of them is an integer in those
 * units; it is kept as a plain little-endian array of 32-bit limbs (72
 * limbs hold 2^2304 units, far above any sum of finite doubles). */
#define EX_LIMBS 72
typedef struct {
    uint32_t w[EX_LIMBS];
} exact_t;

static void ex_zero(exact_t *a) { memset(a->w, 0, sizeof a->w); }

/* a += v * 2^(32 * limb), v < 2^96 given as three 32-bit words */
static void ex_add_at(exact_t *a, int limb, uint64_t lo64, uint32_t hi32)
{
    uint64_t carry = 0;
    uint32_t part[3] = {(uint32_t)lo64, (uint32_t)(lo64 >> 32), hi32};
    for (int i = limb; i < EX_LIMBS; i++) {
        uint64_t add = i - limb < 3 ? part[i - limb] : 0;
        if (i - limb >= 3 && carry == 0)
            break;
        uint64_t t = (uint64_t)a->w[i] + add + carry;
        a->w[i] = (uint32_t)t;
        carry = t >> 32;
    }
}

/* a += x, x finite and >= 0: x = mant * 2^(pos - 1074) with the 53-bit
 * mantissa (implicit bit included for normal numbers) */
static void ex_add_double(exact_t *a, double x)
{
    uint64_t bits;
    memcpy(&bits, &x, sizeof bits);
    int e = (int)(bits >> 52);
    uint64_t mant = bits & ((1ull << 52) - 1);
    int pos = 0;
    if (e > 0) {
        mant |= 1ull << 52;
        pos = e - 1;
    }
    if (mant == 0)
        return;
    int limb = pos / 32, sh = pos % 32;
    /* mant << sh < 2^85: low 64 bits and the bits above */
    uint64_t lo = sh ? mant << sh : mant;
    uint32_t hi = sh ? (uint32_t)(mant >> (64 - sh)) : 0;
    ex_add_at(a, limb, lo, hi);
}

static void ex_add(exact_t *a, const exact_t *b)
{
    uint64_t carry = 0;
    for (int i = 0; i < EX_LIMBS; i++) {
        uint64_t t = (uint64_t)a->w[i] + b->w[i] + carry;
        a->w[i] = (uint32_t)t;
        carry = t >> 32;
    }
}

/* a - b for a >= b */
static void ex_sub(exact_t *d, const exact_t *a, const exact_t *b)
{
    int64_t borrow = 0;
    for (int i = 0; i < EX_LIMBS; i++) {
        int64_t t = (int64_t)a->w[i] - b->w[i] - borrow;
        borrow = t < 0;
        d->w[i] = (uint32_t)(t + (borrow ? (int64_t)1 << 32 : 0));
    }
}

static int ex_cmp(const exact_t *a, const exact_t *b)
{
    for (int i = EX_LIMBS - 1; i >= 0; i--)
        if (a->w[i] != b->w[i])
            return a->w[i] < b->w[i] ? -1 : 1;
    return 0;
}

static int ex_bit(const exact_t *a, int k) { return (a->w[k / 32] >> (k % 32)) & 1u; }

/* the nearest double to a (ties to even); +infinity beyond the largest */
static double ex_round(const exact_t *a)
{
    int top = -1;
    for (int k = 32 * EX_LIMBS - 1; k >= 0; k--)
        if (ex_bit(a, k)) {
            top = k;
            break;
        }
    uint64_t bits;
    if (top < 53) {
        /* below 2^53 units the value is exact: a denormal, or the smallest
         * normal binade, whose encoding is the unit count itself */
        bits = 0;
        for (int k = top; k >= 0; k--)
            bits = bits << 1 | (uint64_t)ex_bit(a, k);
    } else {
        uint64_t m53 = 0;
        for (int k = top; k > top - 53; k--)
            m53 = m53 << 1 | (uint64_t)ex_bit(a, k);
        int half = ex_bit(a, top - 53), sticky = 0;
        for (int k = top - 54; k >= 0 && !sticky; k--)
            sticky = ex_bit(a, k);
        if (half && (sticky || (m53 & 1))) {
            m53++;
            if (m53 == 1ull << 53) {
                m53 >>= 1;
                top++;
            }
        }
        int64_t expo = (int64_t)top - 51; /* value = m53 / 2^52 * 2^(top - 1074) */
        if (expo >= 2047)
            bits = 0x7FFull << 52;
        else
            bits = (uint64_t)expo << 52 | (m53 & ((1ull << 52) - 1));
    }
    double x;
    memcpy(&x, &bits, sizeof x);
    return x;
}

/* Eq. (6) exactly: the sum over (b, m) of the rounded terms (R26) */
static void objective_exact(int32_t n, int32_t m, const double *lam,
                            const double *w, const double *f, const uint8_t *tgt,
                            exact_t *g)
{
    ex_zero(g);
    for (int32_t b = 0; b < n; b++)
        for (int32_t r = 0; r < m; r++) {
            double best = 0.0;
            for (int32_t h = 0; h < m; h++)
                if (tgt[(size_t)h * n + b])
                    best = maxd(best, q_save_f64(n, m, w, f, h, r, b));
            double term = lam[(size_t)r * n + b] * best;
            ex_add_double(g, term);
        }
}

static double objective_f64(int32_t n, int32_t m, const double *lam,
                            const double *w, const double *f, const uint8_t *tgt)
{
    exact_t g;
    objective_exact(n, m, lam, w, f, tgt, &g);
    return ex_round(&g);
}

/* Eq. (7), requester terms in increasing m */
static void marginal_f64(int32_t n, int32_t m, const double *lam,
                         const double *w, const double *f, const uint8_t *tgt,
                         int32_t h, double *profit)
{
    for (int32_t b = 0; b < n; b++) {
        double p = 0.0;
        for (int32_t r = 0; r < m; r++) {
            double v = 0.0;
            for (int32_t l = 0; l < m; l++)
                if (l != h && tgt[(size_t)l * n + b])
                    v = maxd(v, q_save_f64(n, m, w, f, l, r, b));
            double gap = q_save_f64(n, m, w, f, h, r, b) - v;
            double term = lam[(size_t)r * n + b] * maxd(gap, 0.0);
            p += term;
        }
        profit[b] = p;
    }
}

/* Eq. (9) on doubles: the full table, take only if strictly better */
static int rooted_dp_pos_f64(int32_t n, const int32_t *nextpos,
                             const double *profit_pos, int32_t k,
                             uint8_t *sel_pos, double *value)
{
    int64_t kk = k < n ? k : n;
    memset(sel_pos, 0, (size_t)n);
    if (kk <= 0) {
        *value = 0.0;
        return PPO_OK;
    }
    size_t W = (size_t)kk + 1;
    double *D = calloc(((size_t)n + 2) * W, sizeof(double));
    if (!D)
        return PPO_E_NOMEM;
#define CELL(i, j) D[(size_t)(i) * W + (size_t)(j)]
    for (int64_t i = n; i >= 1; i--) {
        int64_t nx = (int64_t)nextpos[i - 1] + 1;
        double p = profit_pos[i - 1];
        for (int64_t j = 1; j <= kk; j++) {
            double s = CELL(nx, j);
            double t = p + CELL(i + 1, j - 1);
            CELL(i, j) = t > s ? t : s;
        }
    }
    *value = CELL(1, kk);
    int64_t i = 1, j = kk;
    while (i <= n && j > 0) {
        int64_t nx = (int64_t)nextpos[i - 1] + 1;
        double s = CELL(nx, j);
        double t = profit_pos[i - 1] + CELL(i + 1, j - 1);
        if (t > s) {
            sel_pos[i - 1] = 1;
            i += 1;
            j -= 1;
        } else {
            i = nx;
        }
    }
#undef CELL
    free(D);
    return PPO_OK;
}

int ppo_rooted_dp_f64(int32_t n, const int32_t *parent, const double *profit,
                      int32_t k, uint8_t *sel, double *value)
{
    if (n < 1 || !parent || !profit || !sel || !value || k < 0)
        return PPO_E_ARG;
    for (int32_t v = 0; v < n; v++)
        if (!finite_nonneg(profit[v]))
            return PPO_E_RANGE;
    int32_t *order = malloc((size_t)n * sizeof(int32_t));
    int32_t *nextpos = malloc((size_t)n * sizeof(int32_t));
    double *pp = malloc((size_t)n * sizeof(double));
    uint8_t *sp = malloc((size_t)n);
    int rc = PPO_E_NOMEM;
    if (!order || !nextpos || !pp || !sp)
        goto out;
    rc = preorder(n, parent, order, nextpos);
    if (rc != PPO_OK)
        goto out;
    for (int32_t i = 0; i < n; i++)
        pp[i] = profit[order[i]];
    rc = rooted_dp_pos_f64(n, nextpos, pp, k, sp, value);
    if (rc == PPO_OK)
        for (int32_t i = 0; i < n; i++)
            sel[order[i]] = sp[i];
out:
    free(order); free(nextpos); free(pp); free(sp);
    return rc;
}

int ppo_marginal_f64(int32_t n, int32_t m, const double *demand,
                     const double *recompute_cost, const double *fetch_cost,
                     const uint8_t *target, int32_t h, double *profit)
{
    if (n < 1 || m < 1 || h < 0 || h >= m || !demand || !recompute_cost ||
        !fetch_cost || !target || !profit)
        return PPO_E_ARG;
    marginal_f64(n, m, demand, recompute_cost, fetch_cost, target, h, profit);
    return PPO_OK;
}

int ppo_objective_f64(int32_t n, int32_t m, const double *demand,
                      const double *recompute_cost, const double *fetch_cost,
                      const uint8_t *target, double *objective)
{
    if (n < 1 || m < 1 || !demand || !recompute_cost || !fetch_cost ||
        !target || !objective)
        return PPO_E_ARG;
    *objective = objective_f64(n, m, demand, recompute_cost, fetch_cost, target);
    return PPO_OK;
}

typedef struct {
    int32_t n, m;
    const double *lam, *w, *f;
    const int32_t *cap;
    const int32_t *order, *nextpos;
    int32_t max_rounds;
    uint32_t flags;
    double eps;
} plan_in_f64;

static int worker_update_f64(const plan_in_f64 *in, const uint8_t *tgt,
                             int32_t h, double *profit, double *pp,
                             uint8_t *sp, uint8_t *cand, double *dpval)
{
    int32_t n = in->n;
    marginal_f64(n, in->m, in->lam, in->w, in->f, tgt, h, profit);
    for (int32_t i = 0; i < n; i++)
        pp[i] = profit[in->order[i]];
    int rc = rooted_dp_pos_f64(n, in->nextpos, pp, in->cap[h], sp, dpval);
    if (rc != PPO_OK)
        return rc;
    for (int32_t i = 0; i < n; i++)
        cand[in->order[i]] = sp[i];
    return PPO_OK;
}

/* Algorithm 1, one start, with the tolerance epsilon of the refinement test */
static int run_start_f64(const plan_in_f64 *in, const int32_t *pi,
                         uint8_t *tgt, exact_t *obj, int32_t *sweeps,
                         int32_t *accepts)
{
    int32_t n = in->n, m = in->m;
    double *profit = malloc((size_t)n * sizeof(double));
    double *pp = malloc((size_t)n * sizeof(double));
    uint8_t *sp = malloc((size_t)n);
    uint8_t *cand = malloc((size_t)n);
    uint8_t *old = malloc((size_t)n);
    int rc = PPO_E_NOMEM;
    if (!profit || !pp || !sp || !cand || !old)
        goto out;
    memset(tgt, 0, (size_t)m * n);
    double v;
    for (int32_t a = 0; a < m; a++) {
        int32_t h = pi[a];
        rc = worker_update_f64(in, tgt, h, profit, pp, sp, cand, &v);
        if (rc != PPO_OK)
            goto out;
        memcpy(tgt + (size_t)h * n, cand, (size_t)n);
    }
    int32_t r = 0, acc = 0;
    if (!(in->flags & PPO_F_NO_REFINE)) {
        int improved;
        do {
            improved = 0;
            for (int32_t a = 0; a < m; a++) {
                int32_t h = pi[a];
                exact_t g_old, g_new, bar;
                objective_exact(n, m, in->lam, in->w, in->f, tgt, &g_old);
                uint8_t *th = tgt + (size_t)h * n;
                memcpy(old, th, (size_t)n);
                memset(th, 0, (size_t)n);
                rc = worker_update_f64(in, tgt, h, profit, pp, sp, cand, &v);
                if (rc != PPO_OK)
                    goto out;
                memcpy(th, cand, (size_t)n);
                objective_exact(n, m, in->lam, in->w, in->f, tgt, &g_new);
                ex_zero(&bar);  /* G(T) + epsilon, exactly */
                ex_add_double(&bar, in->eps);
                ex_add(&bar, &g_old);
                if (ex_cmp(&g_new, &bar) > 0) {
                    improved = 1;
                    acc++;
                } else {
                    memcpy(th, old, (size_t)n);
                }
            }
            r++;
        } while (improved && !(in->max_rounds > 0 && r == in->max_rounds));
    }
    objective_exact(n, m, in->lam, in->w, in->f, tgt, obj);
    *sweeps = r;
    *accepts = acc;
    rc = PPO_OK;
out:
    free(profit); free(pp); free(sp); free(cand); free(old);
    return rc;
}

/* R18 on doubles: fetch_cost[src][dst][b] equal (as values) over src != dst */
static int requester_side_f64(int32_t n, int32_t m, const double *fetch_cost)
{
    for (int32_t dst = 0; dst < m; dst++) {
        int32_t first = dst == 0 ? 1 : 0;
        for (int32_t src = first + 1; src < m; src++) {
            if (src == dst)
                continue;
            for (int32_t b = 0; b < n; b++)
                if (fetch_cost[((size_t)src * m + dst) * n + b] !=
                    fetch_cost[((size_t)first * m + dst) * n + b])
                    return 0;
        }
    }
    return 1;
}

/* The comparator placements (R19) on doubles, with the integer path's
 * formulas: Independent p = Lambda_h * w_h, Popularity p = Lambda_h,
 * LocalDedup p = a + [b not in U] * Lambda_h * [w_h - f_h]_+ with
 * a = Lambda_h * min(w_h, f_h) (M = 1: Lambda_h * w_h). */
static int candidates_f64(int32_t n, int32_t m, const int32_t *order,
                          const int32_t *nextpos, const double *demand,
                          const double *recompute_cost, const double *fetch_cost,
                          const int32_t *cap, uint8_t *targets, exact_t *objs)
{
    double *pp = malloc((size_t)n * sizeof(double));
    uint8_t *sp = malloc((size_t)n);
    int rc = PPO_E_NOMEM;
    if (!pp || !sp)
        goto out;
    memset(targets, 0, (size_t)3 * m * n);
    for (int32_t c = 0; c < 3; c++) {
        uint8_t *tg = targets + (size_t)c * m * n;
        for (int32_t h = 0; h < m; h++) {
            const double *lam = demand + (size_t)h * n;
            const double *w = recompute_cost + (size_t)h * n;
            int32_t src = h == 0 ? 1 : 0;
            const double *f = m > 1 ? fetch_cost + ((size_t)src * m + h) * n : NULL;
            for (int32_t i = 0; i < n; i++) {
                int32_t b = order[i];
                double p;
                if (c == 0) {
                    p = lam[b] * w[b];
                } else if (c == 1) {
                    p = lam[b];
                } else if (!f) {
                    p = lam[b] * w[b];
                } else {
                    int covered = 0;
                    for (int32_t l = 0; l < h; l++)
                        covered |= tg[(size_t)l * n + b];
                    double a = lam[b] * (w[b] < f[b] ? w[b] : f[b]);
                    double own = lam[b] * maxd(w[b] - f[b], 0.0);
                    p = covered ? a : a + own;
                }
                pp[i] = p;
            }
            double v;
            rc = rooted_dp_pos_f64(n, nextpos, pp, cap[h], sp, &v);
            if (rc != PPO_OK)
                goto out;
            for (int32_t i = 0; i < n; i++)
                tg[(size_t)h * n + order[i]] = sp[i];
        }
        objective_exact(n, m, demand, recompute_cost, fetch_cost, tg, &objs[c]);
    }
    rc = PPO_OK;
out:
    free(pp); free(sp);
    return rc;
}

/* The planner on real-valued costs (R24), one start after another.
 * Arguments as ppo_plan, with double inputs and outputs, the tolerance
 * `epsilon` (finite, >= 0), info[5] = {returned candidate (start s, or
 * S + c for safeguard c), updates, DP cells, S, safeguards run} and
 * safeguard_obj[3] (0 if not run). */
int ppo_plan_f64(int32_t n, int32_t m, const int32_t *parent,
                 const double *demand, const double *recompute_cost,
                 const double *fetch_cost, const int32_t *cap, double epsilon,
                 int32_t n_starts, int32_t max_rounds, uint64_t order_seed,
                 const int32_t *orders_in, uint32_t flags, uint8_t *target,
                 double *objective, double *standalone_out,
                 int32_t *orders_out, double *start_objective,
                 int32_t *start_sweeps, int32_t *start_accepts, int64_t *info,
                 double *safeguard_obj)
{
    int rc = validate_f64(n, m, parent, demand, recompute_cost, fetch_cost, cap);
    if (rc != PPO_OK)
        return rc;
    if (n_starts < 0 || max_rounds < 0 || !target || !objective ||
        !finite_nonneg(epsilon))
        return PPO_E_ARG;
    int32_t S = ppo_num_starts(m, n_starts);
    if (orders_in) {
        if (n_starts < 1)
            return PPO_E_ARG;
        for (int32_t s = 0; s < S; s++) {
            uint8_t seen[256] = {0};
            for (int32_t a = 0; a < m; a++) {
                int32_t h = orders_in[(size_t)s * m + a];
                if (h < 0 || h >= m || seen[h])
                    return PPO_E_ARG;
                seen[h] = 1;
            }
        }
    }
    int32_t *order = malloc((size_t)n * sizeof(int32_t));
    int32_t *nextpos = malloc((size_t)n * sizeof(int32_t));
    int32_t *orders = malloc((size_t)S * m * sizeof(int32_t));
    double *standalone = malloc((size_t)m * sizeof(double));
    int64_t *rank = malloc((size_t)m * sizeof(int64_t));
    uint8_t *tgts = malloc((size_t)S * m * n);
    exact_t *obj = calloc((size_t)S, sizeof(exact_t));
    int32_t *sw = malloc((size_t)S * sizeof(int32_t));
    int32_t *ac = malloc((size_t)S * sizeof(int32_t));
    double *profit = malloc((size_t)n * sizeof(double));
    double *pp = malloc((size_t)n * sizeof(double));
    uint8_t *sp = malloc((size_t)n);
    uint8_t *cand = malloc((size_t)n);
    uint8_t *empty = calloc((size_t)m * n, 1);
    uint8_t *cands = NULL;
    rc = PPO_E_NOMEM;
    if (!order || !nextpos || !orders || !standalone || !rank || !tgts ||
        !obj || !sw || !ac || !profit || !pp || !sp || !cand || !empty)
        goto out;
    rc = preorder(n, parent, order, nextpos);
    if (rc != PPO_OK)
        goto out;
    plan_in_f64 in = {n, m, demand, recompute_cost, fetch_cost, cap, order,
                      nextpos, max_rounds, flags, epsilon};
    for (int32_t h = 0; h < m; h++) {  /* R6 */
        rc = worker_update_f64(&in, empty, h, profit, pp, sp, cand,
                               &standalone[h]);
        if (rc != PPO_OK)
            goto out;
    }
    if (orders_in) {
        memcpy(orders, orders_in, (size_t)S * m * sizeof(int32_t));
    } else {
        /* order 0 sorts by score: give equal scores equal integer keys */
        for (int32_t h = 0; h < m; h++) {
            rank[h] = 0;
            for (int32_t l = 0; l < m; l++)
                if (standalone[l] < standalone[h])
                    rank[h]++;
        }
        rc = ppo_orders(m, n_starts, order_seed, rank, orders);
        if (rc != PPO_OK)
            goto out;
    }
    for (int32_t s = 0; s < S; s++) {
        rc = run_start_f64(&in, orders + (size_t)s * m, tgts + (size_t)s * m * n,
                           &obj[s], &sw[s], &ac[s]);
        if (rc != PPO_OK)
            goto out;
    }
    int32_t best = 0;  /* R10, R26: exact values, earliest start on ties */
    for (int32_t s = 1; s < S; s++)
        if (ex_cmp(&obj[s], &obj[best]) > 0)
            best = s;
    const uint8_t *won = tgts + (size_t)best * m * n;
    exact_t won_obj = obj[best];
    exact_t sg_ex[3];
    double sg_obj[3] = {0.0, 0.0, 0.0};
    int sg_run = 0;
    if ((flags & PPO_F_SAFEGUARDS) && requester_side_f64(n, m, fetch_cost)) {
        cands = malloc((size_t)3 * m * n);
        rc = PPO_E_NOMEM;
        if (!cands)
            goto out;
        rc = candidates_f64(n, m, order, nextpos, demand, recompute_cost,
                            fetch_cost, cap, cands, sg_ex);
        if (rc != PPO_OK)
            goto out;
        sg_run = 1;
        for (int32_t c = 0; c < 3; c++) {  /* R20 */
            sg_obj[c] = ex_round(&sg_ex[c]);
            if (ex_cmp(&sg_ex[c], &won_obj) > 0) {
                won_obj = sg_ex[c];
                won = cands + (size_t)c * m * n;
                best = S + c;
            }
        }
    }
    memcpy(target, won, (size_t)m * n);
    *objective = ex_round(&won_obj);
    int64_t updates = m, cells = 0;
    for (int32_t h = 0; h < m; h++)
        cells += (int64_t)n * (cap[h] < n ? cap[h] : n);
    int64_t cells_per_pass = cells;
    for (int32_t s = 0; s < S; s++) {
        updates += (int64_t)m * (1 + sw[s]);
        cells += cells_per_pass * (1 + sw[s]);
    }
    if (standalone_out)
        memcpy(standalone_out, standalone, (size_t)m * sizeof(double));
    if (orders_out)
        memcpy(orders_out, orders, (size_t)S * m * sizeof(int32_t));
    if (start_objective)
        for (int32_t s = 0; s < S; s++)
            start_objective[s] = ex_round(&obj[s]);
    if (start_sweeps)
        memcpy(start_sweeps, sw, (size_t)S * sizeof(int32_t));
    if (start_accepts)
        memcpy(start_accepts, ac, (size_t)S * sizeof(int32_t));
    if (sg_run) {
        updates += 3 * (int64_t)m;
        cells += 3 * cells_per_pass;
    }
    if (info) {
        info[0] = best;
        info[1] = updates;
        info[2] = cells;
        info[3] = S;
        info[4] = sg_run;
    }
    if (safeguard_obj)
        memcpy(safeguard_obj, sg_obj, sizeof sg_obj);
    rc = PPO_OK;
out:
    free(order); free(nextpos); free(orders); free(standalone); free(rank);
    free(tgts); free(obj); free(sw); free(ac); free(profit); free(pp); free(sp);
    free(cand); free(empty); free(cands);
    return rc;
}

/* R21/R22 on doubles: the one-time cost, summed exactly (R26); adoption
 * iff horizon * (G(T') - G(T)) > cost on the rounded exact values. */
static void materialization_cost_exact(int32_t n, int32_t m, const double *w,
                                       const double *f, const uint8_t *incumbent,
                                       const uint8_t *proposal, exact_t *total)
{
    ex_zero(total);
    for (int32_t r = 0; r < m; r++)
        for (int32_t b = 0; b < n; b++) {
            if (!proposal[(size_t)r * n + b] || incumbent[(size_t)r * n + b])
                continue;
            double c = w[(size_t)r * n + b];
            for (int32_t h = 0; h < m; h++)
                if (h != r && incumbent[(size_t)h * n + b]) {
                    double fh = f[((size_t)h * m + r) * n + b];
                    if (fh < c)
                        c = fh;
                }
            ex_add_double(total, c);
        }
}

/* Epoch re-planning on real-valued costs: arguments as ppo_replan, with
 * double inputs, a real horizon (finite, >= 0) and the tolerance epsilon of
 * the planner; result[3] = {G(incumbent), G(proposal), cost}, *adopt. */
int ppo_replan_f64(int32_t n, int32_t m, const int32_t *parent,
                   const double *demand, const double *recompute_cost,
                   const double *fetch_cost, const int32_t *cap,
                   const uint8_t *incumbent, double horizon, double epsilon,
                   int32_t n_starts, int32_t max_rounds, uint64_t order_seed,
                   uint32_t flags, uint8_t *target, uint8_t *proposal,
                   int32_t *adopt, double *result)
{
    if (!incumbent || !target || !result || !adopt || !finite_nonneg(horizon))
        return PPO_E_ARG;
    int rc = validate_f64(n, m, parent, demand, recompute_cost, fetch_cost, cap);
    if (rc != PPO_OK)
        return rc;
    for (size_t x = 0; x < (size_t)m * n; x++)
        if (incumbent[x] > 1)
            return PPO_E_ARG;
    uint8_t *prop = malloc((size_t)m * n);
    if (!prop)
        return PPO_E_NOMEM;
    double g_new;
    rc = ppo_plan_f64(n, m, parent, demand, recompute_cost, fetch_cost, cap,
                      epsilon, n_starts, max_rounds, order_seed, NULL, flags,
                      prop, &g_new, NULL, NULL, NULL, NULL, NULL, NULL, NULL);
    if (rc != PPO_OK) {
        free(prop);
        return rc;
    }
    exact_t e_inc, e_new, e_cost, diff;
    objective_exact(n, m, demand, recompute_cost, fetch_cost, incumbent, &e_inc);
    objective_exact(n, m, demand, recompute_cost, fetch_cost, prop, &e_new);
    materialization_cost_exact(n, m, recompute_cost, fetch_cost, incumbent, prop,
                               &e_cost);
    double gain;  /* G(T') - G(T), exact, then rounded */
    if (ex_cmp(&e_new, &e_inc) >= 0) {
        ex_sub(&diff, &e_new, &e_inc);
        gain = ex_round(&diff);
    } else {
        ex_sub(&diff, &e_inc, &e_new);
        gain = -ex_round(&diff);
    }
    double g_inc = ex_round(&e_inc);
    double cost = ex_round(&e_cost);
    int a = horizon * gain > cost;
    memcpy(target, a ? prop : incumbent, (size_t)m * n);
    if (proposal)
        memcpy(proposal, prop, (size_t)m * n);
    *adopt = a;
    result[0] = g_inc;
    result[1] = g_new;
    result[2] = cost;
    free(prop);
    return PPO_OK;
}
