/*
 * prefixplace.h -- C ABI of the MI355X (gfx950) PrefixPlace planner hot path.
 *
 * PrefixPlace (arXiv 2608.01655) assigns every LLM-serving worker a
 * prefix-complete (parent-closed) set of KV-cache chunks under a per-worker
 * chunk budget, maximising the materialisation cost saved per epoch.
 *
 * Problem (Eq. 8): maximise F_pair(T) (Eq. 6) over T = (T_1..T_M) with
 * |T_m| <= k_m and every T_m parent-closed, where requester m saves
 *   q_{m<-h}(b) = w_m(b)                     if h == m,
 *                 max(w_m(b) - f_{m<-h}(b), 0) otherwise      (Eq. 5)
 * on chunk b when holder h is its best resident copy.  Each worker update
 * computes the exact marginals p_h(b) of Proposition 1 (Eq. 7) and solves
 * the rooted-tree knapsack of Eq. 9 / Theorem 1 exactly; updates run as
 * WorkerGreedy (Theorem 3) followed by coordinate refinement over
 * order-diverse starts (Sec. IV-C, Algorithm 1).
 *
 * Conventions shared by every entry point
 *   - Values: the integer entry points take demand in requests per epoch
 *     and costs in integer microseconds, and every value/objective is int64
 *     (request * us), exact.  The *_f64 entry points take finite,
 *     non-negative IEEE doubles in any consistent units and a refinement
 *     tolerance epsilon >= 0; every objective value they compare is the
 *     exact sum of its rounded terms, so no result depends on an order of
 *     summation.
 *   - Node ids are the caller's labels 0..n-1.  parent[v] = -1 attaches v to
 *     the implicit no-cost dummy root (Sec. III-A), so forests are allowed.
 *   - Host arrays are C-contiguous, caller-owned, read or written only during
 *     the call; the library keeps no pointer after returning.
 *   - On any error the outputs are left unmodified, a negative PP_E_* code is
 *     returned and pp_last_error() describes it.  No C++ exception crosses
 *     this ABI.  Inputs are validated before any device work.
 *   - Tie rules (deterministic):
 *       DP ties keep the skip branch (a node is taken only if strictly
 *       better), so among optimal sets the one whose 0/1 vector in canonical
 *       preorder (roots, then children, by increasing id) is
 *       lexicographically smallest is returned;
 *       a refinement replacement is accepted only if it raises the
 *       objective strictly (integer costs) or by more than epsilon (the
 *       *_f64 entry points);
 *       ties between starts go to the lowest start index.
 *   - Start orders: start 0 sorts workers by standalone score (the optimum
 *     of the worker's own rooted-tree problem against an empty placement)
 *     descending, ties by lower worker id; start 1 is its reverse; start
 *     s >= 2 is a Fisher-Yates shuffle of 0..m-1 driven by SplitMix64
 *     seeded with order_seed + s (j = next() mod (i+1), for i = m-1..1).
 *   - All GPU entry points run on the current HIP device.
 */
#ifndef PREFIXPLACE_H
#define PREFIXPLACE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PP_ABI_VERSION 11

enum {
    PP_OK = 0,
    PP_E_ARG = -1,      /* null pointer, n < 1, m < 1 or m > 255, bad option */
    PP_E_TREE = -2,     /* parent out of range, self-parent, or a cycle */
    PP_E_RANGE = -3,    /* negative demand, cost, capacity or profit */
    PP_E_OVERFLOW = -4, /* sum over (m,b) of demand*recompute exceeds INT64_MAX */
    PP_E_NOMEM = -5,    /* host or device allocation failed */
    PP_E_DEVICE = -6,   /* HIP error, no device, or a device-side stall */
    PP_E_UNSUPPORTED = -7 /* a shape beyond a documented limit (see below) */
};

enum {
    PP_F_VALIDATE_ONLY = 1u, /* validate and build the tree layout, no GPU work */
    PP_F_NO_REFINE = 2u,     /* greedy pass only (Theorem 3's WorkerGreedy) */
    PP_F_TIME_KERNELS = 4u,  /* time every DP-sweep launch with HIP events */
    PP_F_SAFEGUARDS = 8u     /* comparator safeguards (Sec. IV-C, Algorithm 1):
                                when every fetch_cost[src][dst][b], src != dst,
                                is equal over src (requester-side costs; M = 1
                                counts as such), also solve the Independent
                                (p = Lambda_m w_m per worker), Popularity
                                (p = Lambda_m) and LocalDedup (workers in
                                increasing id, p = a_m(b) + 1{b not in U}
                                Lambda_m [w_m - f_m]_+, U = the earlier
                                workers' sets) placements, each a rooted-tree
                                DP per worker, and return one of them if its
                                objective is strictly higher than every
                                start's (ties: Independent, Popularity,
                                LocalDedup).  3M more DP updates.  No effect
                                for source-dependent costs. */
};

/* Planner options.  Passing NULL selects
 * {n_starts = 8, max_rounds = 0, order_seed = 0, orders = NULL, flags = 0}. */
typedef struct {
    int32_t n_starts;       /* >= 1: number of starts; 0: the paper's default
                               set (m <= 5: all m! orders in lexicographic
                               order; otherwise 8 starts) */
    int32_t max_rounds;     /* cap on refinement sweeps, counting the final
                               non-improving one; 0 = until a sweep accepts
                               nothing */
    uint64_t order_seed;    /* seeds the shuffled starts (index >= 2) */
    const int32_t *orders;  /* optional [n_starts][m] explicit worker orders
                               (host); NULL = generate as described above */
    uint32_t flags;         /* PP_F_* */
} pp_options;

/* Optional statistics.  Pointer fields may be NULL; arrays indexed by start
 * must hold pp_num_starts(m, n_starts) entries. */
typedef struct {
    int32_t best_start;        /* out: start whose placement is returned, or
                                  n_starts + c when safeguard candidate c
                                  (0 Independent, 1 Popularity, 2 LocalDedup)
                                  is returned */
    int32_t n_starts;          /* out: number of starts run */
    int64_t updates;           /* out: worker updates of Algorithm 1
                                  (standalone + greedy + every sweep) */
    int64_t dp_cells;          /* out: sum over updates of n * min(k_h, n) */
    int64_t *start_objective;  /* out [S]: objective of each start */
    int32_t *start_sweeps;     /* out [S]: refinement sweeps per start */
    int32_t *start_accepts;    /* out [S]: accepted replacements per start */
    int64_t *standalone;       /* out [m]: standalone score per worker */
    int32_t *orders;           /* out [S][m]: start orders used */
    double dp_kernel_ms;       /* out with PP_F_TIME_KERNELS: summed duration
                                  of the DP-sweep launches */
    int32_t dp_launches;       /* out with PP_F_TIME_KERNELS */
    int32_t safeguards_run;    /* out: 1 if the PP_F_SAFEGUARDS candidates were
                                  evaluated (requester-side costs) */
    int64_t safeguard_objective[3]; /* out: their objectives (Independent,
                                  Popularity, LocalDedup), 0 if not run */
    int64_t dp_cells_executed; /* out: DP cells actually swept.  A refinement
                                  update of a worker whose inputs have not
                                  changed since its last sweep (no other
                                  worker's set changed) would find the same
                                  set and reject it; it is resolved as
                                  rejected without a sweep, so this can be
                                  below dp_cells.  Speculative refinement
                                  updates (later positions of a start swept
                                  in the same launch, valid only if the
                                  earlier ones are rejected) that are
                                  discarded add their cells, so it can also
                                  exceed dp_cells.  Results are unaffected. */
    int32_t dp_lane_cells;     /* out: DP cells per lane of the sweep's
                                  compute wave (1, 2 or 4; 0 if no sweep
                                  ran), chosen per plan */
    int32_t dp_fmax;           /* out: 1 if the sweep took the maximum with
                                  one 64-bit float instruction (every value
                                  below 2^62, or real-valued costs), 0 if
                                  with a compare and two selects */
    int32_t dp_restarts;       /* out: times the plan was run again because a
                                  DP sweep stage gave up a bounded wait for
                                  its neighbour (the sweep's stages must be
                                  resident at once; other work on the GPU
                                  can crowd them out): each run uses fewer
                                  stage blocks per launch and longer waits;
                                  after 2 the call fails with PP_E_DEVICE.
                                  Results are unaffected. */
} pp_stats;

/* Number of starts the options select (see pp_options.n_starts). */
int32_t pp_num_starts(int32_t m, int32_t n_starts);

/* Full planner (Algorithm 1 with exact rooted-tree updates; Eq. 8).
 *   parent          [n]      host; -1 = child of the dummy root
 *   demand          [m][n]   host; Lambda_m(b) >= 0 (Sec. III-A)
 *   recompute_cost  [m][n]   host; w_m(b) >= 0 us
 *   fetch_cost      [m][m][n] host; fetch_cost[src][dst][b] = f_{dst<-src}(b)
 *                            >= 0 us; the src == dst plane is ignored.  A
 *                            requester-side cost f_m(b) is given by repeating
 *                            it over src (this reproduces Eq. 4 exactly).
 *   cap             [m]      host; k_m >= 0 chunks (values above n act as n)
 *   opt                      NULL or options
 *   target          [m][n]   host out: 1 iff b is in T_m; each row is
 *                            parent-closed with at most cap[m] ones
 *   objective                host out: F_pair(T) in request * us
 *   stats                    NULL or statistics
 * Limits: the DP sweep keeps pending skip-target rows in LDS slots (their
 * number is at most the tree depth; 14 and 17 on the 50,000-chunk benchmark
 * trees).  Up to 254 stay in LDS; a deeper tree that branches along long
 * chains has its long-lived pending rows spilled to device memory and
 * restored ahead of their reads (pp_sweep_spills), so any depth is
 * accepted; PP_E_UNSUPPORTED only if even then more than 254 LDS rows would
 * be needed at once, or the rows do not fit one compute unit's LDS. */
int pp_plan(int32_t n, int32_t m, const int32_t *parent, const int64_t *demand,
            const int64_t *recompute_cost, const int64_t *fetch_cost,
            const int32_t *cap, const pp_options *opt, uint8_t *target,
            int64_t *objective, pp_stats *stats);

/* Real-valued costs (the paper's own domain: demand in requests per epoch,
 * costs in milliseconds) with the refinement tolerance epsilon of Algorithm 1
 * (Sec. IV-C): a refinement replacement is accepted only if it raises G by
 * more than epsilon.  Every value is an IEEE double; inputs must be finite
 * and >= 0 (PP_E_RANGE otherwise), epsilon finite and >= 0 (PP_E_ARG).
 * The arithmetic is the integer path's, in doubles: each product
 * Lambda * x is rounded before it is added, p_h(b) adds its requester terms
 * in increasing m, the DP takes b_i only if p + D[i+1][j-1] > D[next(i)][j],
 * and G = F_pair is the exact sum of its rounded terms Lambda_m(b) *
 * max(...) (every finite double is a multiple of 2^-1074, so the sum is kept
 * as an exact integer of those units): a refinement replacement is accepted
 * iff the exact G with it exceeds the exact G(T) + epsilon (so one of
 * exactly equal value, e.g. differing only by chunks of zero marginal value,
 * is never accepted, also at epsilon = 0); starts and comparator candidates
 * compare exact values; reported objectives are the exact values rounded to
 * the nearest double.  PP_F_SAFEGUARDS adds the comparator
 * candidates for requester-side costs (fetch costs equal as values over
 * every source; -0.0 counts as 0.0) with the integer path's formulas in
 * doubles.  Statistics as pp_stats, with double objectives and scores. */
typedef struct {
    int32_t best_start;
    int32_t n_starts;
    int64_t updates;
    int64_t dp_cells;
    double *start_objective;   /* [S] or NULL */
    int32_t *start_sweeps;     /* [S] or NULL */
    int32_t *start_accepts;    /* [S] or NULL */
    double *standalone;        /* [m] or NULL */
    int32_t *orders;           /* [S][m] or NULL */
    double dp_kernel_ms;
    int32_t dp_launches;
    int32_t safeguards_run;
    double safeguard_objective[3];
    int64_t dp_cells_executed;   /* as in pp_stats */
    int32_t dp_lane_cells;       /* as in pp_stats */
    int32_t dp_fmax;             /* as in pp_stats */
    int32_t dp_restarts;         /* as in pp_stats */
} pp_stats_f64;

/* pp_plan on real-valued host arrays (layouts as pp_plan). */
int pp_plan_f64(int32_t n, int32_t m, const int32_t *parent, const double *demand,
                const double *recompute_cost, const double *fetch_cost,
                const int32_t *cap, double epsilon, const pp_options *opt,
                uint8_t *target, double *objective, pp_stats_f64 *stats);

/* pp_rooted_dp on real-valued profits (finite, >= 0). */
int pp_rooted_dp_f64(int32_t n, const int32_t *parent, const double *profit,
                     int32_t k, uint8_t *selected, double *value);

/* Epoch re-planning (Sec. IV-D): when demand or routing changes, plan the
 * refreshed inputs (as pp_plan, same options), evaluate the incumbent under
 * them, and switch to the new plan only when its gain per epoch over the
 * horizon pays for copying in the chunks it newly assigns:
 *   adopt  iff  horizon * (G(T') - G(T)) > sum over (m, b) with b in T'_m
 *               and not in T_m of c_m(b),
 *   c_m(b) = min(w_m(b), min over workers h != m holding b in the
 *            incumbent of f_{m<-h}(b)),
 * G = F_pair (Eq. 6) under the refreshed inputs; the product is compared
 * exactly (no overflow).  Arguments as pp_plan, plus
 *   incumbent [m][n] host: the current placement (0/1; it need not be
 *                    parent-closed or within the new capacities)
 *   horizon          epochs over which the gain is counted (>= 0)
 *   target    [m][n] host out: the placement to use (T' if adopted, else a
 *                    copy of the incumbent)
 *   proposal  [m][n] host out, may be NULL: T'
 *   info             out, required
 * Errors as pp_plan; PP_E_ARG for a negative horizon or an incumbent entry
 * other than 0 and 1, PP_E_OVERFLOW if the one-time cost exceeds INT64_MAX. */
typedef struct {
    int32_t adopt;                 /* 1 iff T' is adopted */
    int64_t incumbent_objective;   /* G(T) under the refreshed inputs */
    int64_t proposal_objective;    /* G(T') */
    int64_t materialization_cost;  /* one-time cost of T' over T, us */
} pp_replan_info;

int pp_replan(int32_t n, int32_t m, const int32_t *parent, const int64_t *demand,
              const int64_t *recompute_cost, const int64_t *fetch_cost,
              const int32_t *cap, const uint8_t *incumbent, int64_t horizon,
              const pp_options *opt, uint8_t *target, uint8_t *proposal,
              pp_replan_info *info, pp_stats *stats);

/* pp_replan on real-valued costs: the planner of pp_plan_f64 (tolerance
 * epsilon), the same rule with a real horizon (finite, >= 0):
 * adopt iff horizon * (G(T') - G(T)) > cost, where G(T') - G(T) and the
 * cost are exact sums each rounded once to the nearest double, and the
 * product and comparison are evaluated in doubles.  Errors as pp_plan_f64
 * and pp_replan. */
typedef struct {
    int32_t adopt;
    double incumbent_objective;
    double proposal_objective;
    double materialization_cost;
} pp_replan_info_f64;

int pp_replan_f64(int32_t n, int32_t m, const int32_t *parent, const double *demand,
                  const double *recompute_cost, const double *fetch_cost,
                  const int32_t *cap, const uint8_t *incumbent, double horizon,
                  double epsilon, const pp_options *opt, uint8_t *target,
                  uint8_t *proposal, pp_replan_info_f64 *info, pp_stats_f64 *stats);

/* One exact rooted-tree solve (Eq. 9, Theorem 1) on the GPU.
 *   parent [n] host, profit [n] host (>= 0, sum <= INT64_MAX), k >= 0;
 *   selected [n] host out (0/1, parent-closed, at most min(k, n) ones);
 *   value host out = max total profit. */
int pp_rooted_dp(int32_t n, const int32_t *parent, const int64_t *profit,
                 int32_t k, uint8_t *selected, int64_t *value);

/* Exact marginals of worker h against the other workers' current sets
 * (Proposition 1, Eq. 7), on the GPU.
 *   target [m][n] host: current placement (row h is ignored);
 *   profit [n] host out: p_h(b);
 *   g_without_h host out (may be NULL): F_pair with T_h emptied. */
int pp_marginal(int32_t n, int32_t m, const int64_t *demand,
                const int64_t *recompute_cost, const int64_t *fetch_cost,
                const uint8_t *target, int32_t h, int64_t *profit,
                int64_t *g_without_h);

/* F_pair(T) of Eq. 6 for an arbitrary placement (target [m][n] host), on
 * the GPU. */
int pp_objective(int32_t n, int32_t m, const int64_t *demand,
                 const int64_t *recompute_cost, const int64_t *fetch_cost,
                 const uint8_t *target, int64_t *objective);

/* Allocation-free F_pair(T), for callers that cannot allocate device memory
 * (code under HIP graph capture set-up, tight serving loops, harnesses that
 * forbid hipMalloc): the value pp_objective returns, on device-resident
 * arrays in caller ids (layouts as pp_plan; target [m][n], a chunk is held
 * where the byte is nonzero), enqueued on `hip_stream` (a hipStream_t; NULL
 * = the null stream).  The call waits for the stream and writes the result
 * to the host `objective`.  It calls no hipMalloc, hipFree or other
 * allocating routine, host or device: its only device memory besides the
 * caller's arrays is a file-scope array of PP_NOALLOC_SCRATCH_BYTES in the
 * library, one per GPU, held until the process ends.  The scratch does not
 * grow with the input (at most 1024 per-block partial sums), so every size
 * pp_objective accepts is accepted: n >= 1, 1 <= m <= 255.  Every call on a
 * GPU shares that GPU's array: calls that overlap on one GPU (other threads,
 * other streams) race and must be serialized by the caller.  Errors as
 * pp_objective: PP_E_ARG (null pointer, sizes), PP_E_RANGE (negative value),
 * PP_E_OVERFLOW (sum of demand * recompute cost above INT64_MAX),
 * PP_E_DEVICE (HIP error); *objective is then left unchanged. */
#define PP_NOALLOC_SCRATCH_BYTES 40960
int pp_objective_device_noalloc(int32_t n, int32_t m, const int64_t *demand_dev,
                                const int64_t *recompute_dev,
                                const int64_t *fetch_dev, const uint8_t *target_dev,
                                int64_t *objective, void *hip_stream);

/* Start orders (Sec. IV-C) from standalone scores [m]; host only.
 * orders [pp_num_starts(m, n_starts)][m] host out. */
int pp_orders(int32_t m, int32_t n_starts, uint64_t order_seed,
              const int64_t *standalone, int32_t *orders);

/* Reusable GPU context: keeps device buffers between calls.  A context is
 * used by one thread at a time; separate contexts may run concurrently. */
typedef struct pp_ctx pp_ctx;
int pp_ctx_create(pp_ctx **ctx, int device);
void pp_ctx_destroy(pp_ctx *ctx);

/* pp_plan with device-resident inputs and output, on `hip_stream`
 * (a hipStream_t; NULL = the null stream).  demand_dev, recompute_dev,
 * fetch_dev are device pointers in caller ids, laid out as in pp_plan;
 * target_dev [m][n] device out.  parent, cap and the options stay on the
 * host.  The call returns after the plan has finished on the stream. */
int pp_plan_device(pp_ctx *ctx, int32_t n, int32_t m, const int32_t *parent,
                   const int64_t *demand_dev, const int64_t *recompute_dev,
                   const int64_t *fetch_dev, const int32_t *cap,
                   const pp_options *opt, uint8_t *target_dev,
                   int64_t *objective, pp_stats *stats, void *hip_stream);

/* pp_plan_device on real-valued device arrays (layouts as pp_plan_device;
 * the value checks run on the device). */
int pp_plan_f64_device(pp_ctx *ctx, int32_t n, int32_t m, const int32_t *parent,
                       const double *demand_dev, const double *recompute_dev,
                       const double *fetch_dev, const int32_t *cap, double epsilon,
                       const pp_options *opt, uint8_t *target_dev, double *objective,
                       pp_stats_f64 *stats, void *hip_stream);

/* Host only, for inspection and CPU-side checks of the DP sweep's step
 * schedule: for the tree `parent` and `cells` (1, 2 or 4) DP cells per
 * lane, writes the per-step metadata of the sweep (`meta`, may be NULL to
 * query the size; 4 * nsteps words, nsteps = n padded up to a multiple of 32
 * with leading dummy steps; step s handles preorder row n - (s - pad), pad =
 * nsteps - n) and the number of LDS slot rows H.  LDS rows hold 64*cells
 * int64 (stride 512*cells + 8 bytes) in the order [H slot rows | zero row |
 * sink rows: 16 at one cell per lane, else 4].  Per step: word 0 = byte
 * offset of the row the step's DP row is stored to (its slot when a later
 * non-leaf row skips to it, else sink row step mod the sink count); word 1 =
 * byte offset of the row read as the next step's skip operand (Eq. 9's
 * D[next(i)][*]: a slot, or the zero row when that next() is past the end or
 * the next step's node is a leaf), which the sweep reads right after storing
 * the current step's row; word 2 = 0xFFFFFFFF when the step's node is a leaf
 * (skip operand: the previous row, in registers), else 0; word 3 = 0.  The
 * first step's node is a leaf. */
int pp_sweep_layout(int32_t n, const int32_t *parent, int32_t cells,
                    uint32_t *meta, int32_t *nsteps, int32_t *slots);

/* Host only, for CPU-side checks of the DP sweep on deep trees.  The sweep
 * keeps each pending skip row (a row that a later non-leaf row reads as its
 * D[next(i)][*]) in an LDS slot; when a tree has more of them pending at
 * once than the slots hold (deep trees that branch along long chains), the
 * rows first read kSpillGap = 3 or more sweep batches (of 32 steps) after
 * their store are spilled: stored to a temporary slot as usual, copied to
 * device memory by the stage's I/O wave once their batch is done (and
 * before it stages the batch after next), and copied back into a restore
 * slot when it stages each later batch that reads them.  Writes nbatches
 * (padded steps / 32), nspill (spill rows per stage; 0 = nothing spilled,
 * then the lists are empty and the offsets zero), n_out and n_in (list
 * entries); each of out_off, spill_out, in_off, spill_in may be NULL.
 * out_off [nbatches + 1]: batch b copies out the entries
 *   spill_out[2e], spill_out[2e + 1] = (LDS slot, spill index) for
 *   e in [out_off[b], out_off[b + 1]);
 * in_off [nbatches + 1]: batch b is staged after copying in the entries
 *   spill_in[2e], spill_in[2e + 1] = (LDS slot, spill index) for
 *   e in [in_off[b], in_off[b + 1]).
 * The step metadata of pp_sweep_layout already names the temporary and
 * restore slots.  Errors as pp_sweep_layout, PP_E_UNSUPPORTED if the
 * pending rows exceed 254 LDS rows even with spilling. */
int pp_sweep_spills(int32_t n, const int32_t *parent, int32_t *nbatches, int32_t *nspill,
                    int32_t *n_out, int32_t *n_in, int32_t *out_off, int32_t *spill_out,
                    int32_t *in_off, int32_t *spill_in);

/* Exit row in pp_backtrack_table for a skip sequence that runs past the
 * last row. */
#define PP_BT_END 0x7FFFFFFFu

/* Host only, for inspection and CPU-side checks of the backtrack's skip
 * table (Theorem 1's walk from (1, k'): a take moves to row i+1, a skip to
 * next(i)).  Rows are 0-based preorder positions, grouped in windows of 32
 * (rows 32w .. 32w+31).  For row q < n, with S(q) = q, next(q),
 * next(next(q)), ... (next(q) = first position after q's subtree):
 *   word 0 = mask of S(q) inside q's window, bit (r mod 32) for each row r
 *            of S(q) below min(32(w+1), n);
 *   word 1 = the first row of S(q) at or past that bound if it is < n, else
 *            PP_BT_END;
 *   word 2 = word 0 of that row (0 for PP_BT_END);
 *   word 3 = 0.
 * Rows n .. rows-1 are padding: {0, PP_BT_END, 0, 0}; rows = n rounded up to
 * a multiple of 512, plus 512.  `table` (4 * rows words) may be NULL to
 * query `rows`.  Errors as for pp_sweep_layout. */
int pp_backtrack_table(int32_t n, const int32_t *parent, uint32_t *table,
                       int64_t *rows);

/* Description of the last error on the calling thread; valid until the
 * next pp_* call on that thread. */
const char *pp_last_error(void);

int pp_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PREFIXPLACE_H */
