// pp_host.cpp -- host side of the PrefixPlace planner: input validation,
// canonical preorder and DP-sweep metadata, start orders, the update loop
// of Algorithm 1 (standalone scores, WorkerGreedy, coordinate refinement,
// best start) and the C ABI of include/prefixplace.h.
//
// Every step of a worker update runs in the gfx950 kernels of
// pp_kernels.hip; this file only prepares layouts and sequences launches.

#include "prefixplace.h"
#include "pp_internal.h"

#include <algorithm>
#include <climits>
#include <cstdlib>
#include <cfloat>
#include <cstring>
#include <memory>
#include <new>
#include <queue>
#include <string>
#include <unordered_map>
#include <vector>

using namespace pp;

namespace {

// Description of the last error on this thread, in a fixed buffer (setting
// it allocates nothing, which the allocation-free entry point relies on).
thread_local char g_err[512];

int fail_c(int code, const char* msg) {
  std::strncpy(g_err, msg, sizeof g_err - 1);
  g_err[sizeof g_err - 1] = 0;
  return code;
}

int fail(int code, const std::string& msg) { return fail_c(code, msg.c_str()); }

// A DP sweep stage gave up a bounded wait (its stages were not all resident
// at once, e.g. with other work on the GPU): the plan is run again with
// fewer stages per launch and a longer wait, up to kStallRetries times.
thread_local bool g_stall = false;
constexpr int kStallRetries = 2;
constexpr uint32_t kDefaultSpin = 1u << 22;

int stall_fail() {
  g_stall = true;
  return fail_c(PP_E_DEVICE, "DP pipeline wait gave up (stages not co-resident)");
}

#define PP_HIP(expr)                                                      \
  do {                                                                    \
    hipError_t e_ = (expr);                                               \
    if (e_ != hipSuccess)                                                 \
      return fail(PP_E_DEVICE, std::string(#expr) + ": " +                \
                                   hipGetErrorString(e_));                \
  } while (0)

#define PP_TRY(expr)            \
  do {                          \
    int rc_ = (expr);           \
    if (rc_ != PP_OK) return rc_; \
  } while (0)

// ------------------------------------------------------------ buffers ---

struct DevBuf {
  void* p = nullptr;
  size_t cap = 0;
  // Grow to at least `bytes`; zero the new memory when `zero`.
  int ensure(size_t bytes, bool zero = false) {
    if (bytes == 0) bytes = 64;
    if (bytes <= cap) return PP_OK;
    if (p) (void)hipFree(p);
    p = nullptr;
    cap = 0;
    if (hipMalloc(&p, bytes) != hipSuccess)
      return fail(PP_E_NOMEM, "device allocation of " + std::to_string(bytes) +
                                  " bytes failed");
    cap = bytes;
    if (zero && hipMemset(p, 0, bytes) != hipSuccess)
      return fail(PP_E_DEVICE, "hipMemset failed");
    return PP_OK;
  }
  void release() {
    if (p) (void)hipFree(p);
    p = nullptr;
    cap = 0;
  }
  template <class T>
  T* as() const { return static_cast<T*>(p); }
};

// --------------------------------------------------------------- tree ---

// Canonical preorder (roots, then children, in increasing id) and the DP
// sweep's per-step metadata.  `order[pos]` is the caller id at 0-based
// position pos, `nextpos[pos]` the first position after its subtree.
struct TreeLayout {
  int32_t n = 0;
  std::vector<int32_t> order, nextpos;
  // the backtrack's skip chains inside 32-row windows [32w, 32w + 32), as
  // ce[4q] = chain mask, ce[4q + 1] = exit row, ce[4q + 2] = the exit row's
  // own chain mask, ce[4q + 3] = 0: the mask has bit r set for every row
  // 32w + r of q, next(q), next(next(q)), ... that lies in q's window; the
  // exit row is the first row of that sequence past the window (kCeEnd if
  // that is past the last row, with mask 0).  Padded with empty rows (mask
  // 0, exit kCeEnd) through one 512-row block past the last full block.
  std::vector<uint32_t> ce;
  // per padded DP step: leaf flag (next(i) = i+1), the LDS slot the row is
  // stored to (-1: a sink row), and the slot holding the next step's skip
  // operand (-1: the zero row, or the next step is a leaf)
  std::vector<uint8_t> leaf;
  std::vector<int32_t> store, src;
  int32_t slots = 0;    // LDS stack rows the sweep needs
  bool identity = true; // caller ids are already in preorder
  // Trees with more pending skip rows than the LDS slots hold (deep trees
  // that branch along long chains): rows whose first read comes at least
  // kSpillGap batches after their store are spilled to device memory.  Per
  // sweep batch b, spill_out[out_off[b] .. out_off[b+1]) lists (LDS slot,
  // spill index) pairs that the I/O wave copies out once batch b is done,
  // and spill_in[in_off[b] .. in_off[b+1]) the (LDS slot, spill index) pairs
  // it copies back in when it stages batch b.  nspill = 0: no spilling.
  std::vector<int32_t> out_off, spill_out, in_off, spill_in;
  int32_t nspill = 0;
};

int layout_sweep(TreeLayout& t);
int layout_sweep_spilled(TreeLayout& t, int32_t pad, int32_t nsteps);

int build_tree(int32_t n, const int32_t* parent, TreeLayout& t) {
  for (int32_t v = 0; v < n; ++v) {
    const int32_t p = parent[v];
    if (p < -1 || p >= n || p == v)
      return fail(PP_E_TREE, "parent[" + std::to_string(v) + "] = " +
                                 std::to_string(p) + " is out of range or self");
  }
  // children in increasing id via counting sort on the parent (roots under
  // the dummy index n)
  std::vector<int32_t> head(n + 2, 0), kids(n);
  for (int32_t v = 0; v < n; ++v) head[(parent[v] < 0 ? n : parent[v]) + 1]++;
  for (int32_t u = 0; u <= n; ++u) head[u + 1] += head[u];
  {
    std::vector<int32_t> fill(head.begin(), head.end() - 1);
    for (int32_t v = 0; v < n; ++v) kids[fill[parent[v] < 0 ? n : parent[v]]++] = v;
  }
  t.n = n;
  t.order.assign(n, 0);
  t.nextpos.assign(n, 0);
  std::vector<int32_t> stack;
  stack.reserve(n);
  for (int32_t k = head[n + 1] - 1; k >= head[n]; --k) stack.push_back(kids[k]);
  int32_t pos = 0;
  std::vector<int32_t> posof(n, -1);
  while (!stack.empty()) {
    const int32_t v = stack.back();
    stack.pop_back();
    posof[v] = pos;
    t.order[pos++] = v;
    for (int32_t k = head[v + 1] - 1; k >= head[v]; --k) stack.push_back(kids[k]);
  }
  if (pos != n) return fail(PP_E_TREE, "parent[] contains a cycle");
  std::vector<int32_t> size(n, 1);
  for (int32_t q = n - 1; q >= 0; --q) {
    const int32_t p = parent[t.order[q]];
    if (p >= 0) size[posof[p]] += size[q];
  }
  t.identity = true;
  for (int32_t q = 0; q < n; ++q) {
    t.nextpos[q] = q + size[q];
    if (t.order[q] != q) t.identity = false;
  }
  const size_t ce_rows = ((size_t)n + kCeBlock - 1) / kCeBlock * kCeBlock + kCeBlock;
  t.ce.assign(4 * ce_rows, 0);
  for (size_t q = n; q < ce_rows; ++q) t.ce[4 * q + 1] = kCeEnd;
  for (int32_t q = n - 1; q >= 0; --q) {
    const int32_t wend = std::min<int32_t>((q / 32 + 1) * 32, n);
    const int32_t nq = t.nextpos[q];  // > q
    uint32_t* e = &t.ce[4 * (size_t)q];
    if (nq < wend) {  // the chain continues inside the window
      e[0] = (1u << (q % 32)) | t.ce[4 * (size_t)nq];
      e[1] = t.ce[4 * (size_t)nq + 1];
      e[2] = t.ce[4 * (size_t)nq + 2];
    } else {
      e[0] = 1u << (q % 32);
      e[1] = nq < n ? (uint32_t)nq : kCeEnd;
      e[2] = nq < n ? t.ce[4 * (size_t)nq] : 0u;
    }
  }
  return layout_sweep(t);
}

// DP metadata.  Rows are 1-based positions i; nx(i) = next(i); row i is
// produced at padded step pad + n - i.  A row r = next(a) with r != a+1
// (a is no leaf) and r != n+1 is a far target: it is stored to an LDS
// slot at its own step, and a reader a reads it right after the store two
// steps before its own.  Every other row is stored to a sink row (step
// mod the sink row count).  Every few steps (the sink row count, at most
// kDpGatherMax) the stage gathers its last cell column from the rows those
// steps were stored to, so a slot becomes free after its last reader (the
// smallest a) has read it and after the gather of its group.
int layout_sweep(TreeLayout& t) {
  const int32_t n = t.n;
  auto nx = [&](int32_t i) { return t.nextpos[i - 1] + 1; };
  auto far = [&](int32_t a, int32_t r) { return r != a + 1 && r != n + 1; };
  std::vector<int32_t> last_user(n + 2, INT32_MAX), slot_of(n + 2, -1);
  for (int32_t a = n; a >= 1; --a) {
    const int32_t r = nx(a);
    if (far(a, r)) last_user[r] = a;  // descending: ends at min
  }
  const int32_t nsteps = (n + kDpBatch - 1) / kDpBatch * kDpBatch;
  const int32_t pad = nsteps - n;
  t.leaf.assign(nsteps, 1);
  t.store.assign(nsteps, -1);
  t.src.assign(nsteps, -1);
  t.out_off.clear();
  t.spill_out.clear();
  t.in_off.clear();
  t.spill_in.clear();
  t.nspill = 0;
  // Free slots as a bitmap (the lowest is taken first), and slots waiting
  // for their release step: a release is due at most kDpGatherMax - 1 steps
  // ahead, so it waits in the bitmap of its step modulo kDpGatherMax.
  static_assert(kMaxSlots <= 256, "slot bitmaps");
  struct Slots {
    uint64_t w[4] = {0, 0, 0, 0};
    void set(int32_t k) { w[k >> 6] |= 1ull << (k & 63); }
    bool any() const { return (w[0] | w[1] | w[2] | w[3]) != 0; }
    int32_t take_lowest() {
      for (int q = 0; q < 4; ++q)
        if (w[q]) {
          const int b = __builtin_ctzll(w[q]);
          w[q] &= w[q] - 1;
          return q * 64 + b;
        }
      return -1;
    }
    void absorb(Slots& o) {
      for (int q = 0; q < 4; ++q) {
        w[q] |= o.w[q];
        o.w[q] = 0;
      }
    }
  };
  Slots free_slots, releases[kDpGatherMax];
  int32_t high = 0;
  bool overflow = false;
  for (int32_t i = n; i >= 1 && !overflow; --i) {
    const int32_t s = pad + n - i;  // padded step of row i
    free_slots.absorb(releases[s % kDpGatherMax]);
    const int32_t r = nx(i);
    t.leaf[s] = (r == i + 1) ? 1 : 0;
    if (far(i, r) && last_user[r] == i) {
      // read at step s-2; written at step s(r), gathered at the end of its
      // group
      const int32_t sr = pad + n - r;
      const int32_t after_gather = (sr / kDpGatherMax + 1) * kDpGatherMax;
      const int32_t at = std::max(s, after_gather);  // < s + kDpGatherMax
      if (at <= s)
        free_slots.set(slot_of[r]);
      else
        releases[at % kDpGatherMax].set(slot_of[r]);
    }
    if (last_user[i] != INT32_MAX) {
      int32_t k;
      if (free_slots.any()) {
        k = free_slots.take_lowest();
      } else {
        if (high >= kMaxSlots) {
          overflow = true;
          break;
        }
        k = high++;
      }
      slot_of[i] = k;
      t.store[s] = k;
    }
    if (i > 1) {
      const int32_t r2 = nx(i - 1);
      if (far(i - 1, r2)) {
        if (slot_of[r2] < 0) return fail(PP_E_DEVICE, "internal: far row without a slot");
        t.src[s] = slot_of[r2];
      }
    }
  }
  if (!overflow) {
    t.slots = high;
    return PP_OK;
  }
  return layout_sweep_spilled(t, pad, nsteps);
}

// The sweep's slots when the pending skip rows do not fit the LDS slots.
// A far target with a read issued kSpillGap or more batches after its store
// is spilled: the compute wave stores it to a temporary slot as usual, which
// also serves the reads issued in the batches before that; the I/O wave
// copies it to device memory once its batch is done (and before it stages
// the batch after next, so the slot is free again two batches on), and
// copies it back into a restore slot when it stages each later batch that
// issues a read of it (at the earliest once the batch two before is done,
// so the restore slot must be free from the start of the batch before).
// The compute wave's schedule is unchanged.  Slots and spill indices are
// assigned by greedy interval colouring (lowest free index first) of their
// lifetimes, half-open step intervals for slots and batch intervals for
// spill indices.
int layout_sweep_spilled(TreeLayout& t, int32_t pad, int32_t nsteps) {
  const int32_t n = t.n;
  const int32_t nb = nsteps / kDpBatch;
  auto nx = [&](int32_t i) { return t.nextpos[i - 1] + 1; };
  auto far = [&](int32_t a, int32_t r) { return r != a + 1 && r != n + 1; };
  auto step_of = [&](int32_t i) { return pad + n - i; };
  auto gather_end = [](int32_t sr) { return (sr / kDpGatherMax + 1) * kDpGatherMax; };
  // a read of row r = next(a) is issued at step (step of a) - 2; its slot
  // is recorded in src[(step of a) - 1]
  std::vector<int32_t> is_target(n + 2, 0), last_early(n + 2, -1), last_issue(n + 2, -1);
  std::vector<uint8_t> spilled(n + 2, 0);
  for (int32_t a = n; a >= 1; --a) {
    const int32_t r = nx(a);
    if (!far(a, r)) continue;
    const int32_t is = step_of(a) - 2, br = step_of(r) / kDpBatch;
    is_target[r] = 1;
    last_issue[r] = std::max(last_issue[r], is);
    if (is / kDpBatch < br + kSpillGap)
      last_early[r] = std::max(last_early[r], is);
    else
      spilled[r] = 1;
  }
  struct Iv {
    int32_t lo, hi;  // live steps [lo, hi)
    int32_t row, batch;
    bool restore;
  };
  std::vector<Iv> iv;
  std::unordered_map<int64_t, size_t> restore_of;  // (row, batch) -> interval
  for (int32_t r = 1; r <= n; ++r) {
    if (!is_target[r]) continue;
    const int32_t sr = step_of(r), br = sr / kDpBatch;
    int32_t hi = std::max(gather_end(sr), last_early[r] + 2);  // the early readers' steps
    if (spilled[r]) hi = std::max(hi, (br + 2) * kDpBatch);
    iv.push_back({sr, hi, r, br, false});
  }
  for (int32_t a = n; a >= 1; --a) {
    const int32_t r = nx(a);
    if (!far(a, r) || !spilled[r]) continue;
    const int32_t is = step_of(a) - 2, b = is / kDpBatch;
    if (b < step_of(r) / kDpBatch + kSpillGap) continue;  // served by the temporary slot
    const int64_t key = (int64_t)r * nb + b;
    auto it = restore_of.find(key);
    if (it != restore_of.end()) {
      iv[it->second].hi = std::max(iv[it->second].hi, is + 1);
    } else {
      restore_of[key] = iv.size();
      iv.push_back({(b - 1) * kDpBatch, is + 1, r, b, true});
    }
  }
  std::vector<size_t> ord(iv.size());
  for (size_t k = 0; k < iv.size(); ++k) ord[k] = k;
  std::stable_sort(ord.begin(), ord.end(),
                   [&](size_t u, size_t v) { return iv[u].lo < iv[v].lo; });
  // interval colouring over at most kMaxSlots slots
  std::vector<int32_t> slot(iv.size(), -1), busy_until;
  for (size_t k : ord) {
    int32_t best = -1;
    for (size_t q = 0; q < busy_until.size(); ++q)
      if (busy_until[q] <= iv[k].lo) {
        best = (int32_t)q;
        break;
      }
    if (best < 0) {
      if ((int32_t)busy_until.size() >= kMaxSlots)
        return fail(PP_E_UNSUPPORTED,
                    "tree needs more than 254 LDS rows for its pending skip rows "
                    "even with spilling");
      best = (int32_t)busy_until.size();
      busy_until.push_back(0);
    }
    busy_until[best] = iv[k].hi;
    slot[k] = best;
  }
  t.slots = (int32_t)busy_until.size();
  // spill indices, live from the store's batch to the last read's batch
  std::vector<int32_t> spill_idx(n + 2, -1);
  {
    std::vector<int32_t> rows;
    for (int32_t r = n; r >= 1; --r)  // increasing store step
      if (spilled[r]) rows.push_back(r);
    using Busy = std::pair<int32_t, int32_t>;  // (last batch, index)
    std::priority_queue<Busy, std::vector<Busy>, std::greater<Busy>> busy;
    std::priority_queue<int32_t, std::vector<int32_t>, std::greater<int32_t>> freed;
    int32_t count = 0;
    for (int32_t r : rows) {
      const int32_t lo = step_of(r) / kDpBatch;
      while (!busy.empty() && busy.top().first < lo) {
        freed.push(busy.top().second);
        busy.pop();
      }
      int32_t k;
      if (!freed.empty()) {
        k = freed.top();
        freed.pop();
      } else {
        k = count++;
      }
      busy.push({last_issue[r] / kDpBatch, k});
      spill_idx[r] = k;
    }
    t.nspill = count;
  }
  // the step schedule and the per-batch copy lists
  std::vector<int32_t> row_slot(n + 2, -1);
  std::vector<std::vector<std::pair<int32_t, int32_t>>> outs(nb), ins(nb);
  for (size_t k = 0; k < iv.size(); ++k) {
    const Iv& v = iv[k];
    if (v.restore) {
      ins[v.batch].push_back({slot[k], spill_idx[v.row]});
    } else {
      row_slot[v.row] = slot[k];
      if (spilled[v.row]) outs[v.batch].push_back({slot[k], spill_idx[v.row]});
    }
  }
  for (int32_t i = n; i >= 1; --i) {
    const int32_t s = step_of(i);
    const int32_t r = nx(i);
    t.leaf[s] = (r == i + 1) ? 1 : 0;
    if (is_target[i]) t.store[s] = row_slot[i];
    if (i > 1) {
      const int32_t r2 = nx(i - 1);
      if (far(i - 1, r2)) {
        const int32_t b = (s - 1) / kDpBatch;  // batch issuing this read
        int32_t k = row_slot[r2];
        if (spilled[r2] && b >= step_of(r2) / kDpBatch + kSpillGap) {
          auto it = restore_of.find((int64_t)r2 * nb + b);
          k = it == restore_of.end() ? -1 : slot[it->second];
        }
        if (k < 0) return fail(PP_E_DEVICE, "internal: far row without a slot");
        t.src[s] = k;
      }
    }
  }
  t.out_off.assign(nb + 1, 0);
  t.in_off.assign(nb + 1, 0);
  for (int32_t b = 0; b < nb; ++b) {
    for (const auto& e : outs[b]) {
      t.spill_out.push_back(e.first);
      t.spill_out.push_back(e.second);
    }
    for (const auto& e : ins[b]) {
      t.spill_in.push_back(e.first);
      t.spill_in.push_back(e.second);
    }
    t.out_off[b + 1] = (int32_t)t.spill_out.size() / 2;
    t.in_off[b + 1] = (int32_t)t.spill_in.size() / 2;
  }
  return PP_OK;
}

// DP-sweep metadata for `cells` cells per lane (layout in pp_internal.h):
// kMetaWords words per padded step.
std::vector<uint32_t> encode_meta(const TreeLayout& t, int cells) {
  const int64_t row = dp_row_stride(cells);  // bytes per LDS row
  const int64_t zero = (int64_t)t.slots * row, sink0 = zero + row;
  const int32_t nsteps = (int32_t)t.leaf.size();
  std::vector<uint32_t> meta(kMetaWords * (size_t)nsteps);
  for (int32_t s = 0; s < nsteps; ++s) {
    uint32_t* w = meta.data() + kMetaWords * (size_t)s;
    w[0] = (uint32_t)(t.store[s] >= 0 ? t.store[s] * row
                                      : sink0 + (s % dp_sink_rows(cells)) * row);
    w[1] = (uint32_t)(t.src[s] >= 0 ? t.src[s] * row : zero);
    w[2] = t.leaf[s] ? 0xFFFFFFFFu : 0u;
    w[3] = 0u;
  }
  return meta;
}

int upload_meta(pp_ctx* c, const TreeLayout& t, int cells, hipStream_t st);
int upload_spills(pp_ctx* c, const TreeLayout& t, DevState& d, int32_t slots,
                  hipStream_t st);

// ------------------------------------------------------------- orders ---

uint64_t splitmix64_next(uint64_t& state) {
  uint64_t z = (state += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

int32_t num_starts(int32_t m, int32_t n_starts) {
  if (n_starts > 0) return n_starts;
  if (m <= 5) {
    int32_t f = 1;
    for (int32_t k = 2; k <= m; ++k) f *= k;
    return f;
  }
  return 8;
}

void make_orders(int32_t m, int32_t n_starts, uint64_t seed,
                 const int64_t* score, int32_t* out) {
  const int32_t S = num_starts(m, n_starts);
  if (n_starts == 0 && m <= 5) {  // every order, lexicographic
    std::vector<int32_t> p(m);
    for (int32_t h = 0; h < m; ++h) p[h] = h;
    for (int32_t s = 0; s < S; ++s) {
      std::copy(p.begin(), p.end(), out + (size_t)s * m);
      std::next_permutation(p.begin(), p.end());
    }
    return;
  }
  std::vector<int32_t> base(m);
  for (int32_t h = 0; h < m; ++h) base[h] = h;
  std::stable_sort(base.begin(), base.end(), [&](int32_t a, int32_t b) {
    return score[a] > score[b];  // stable: equal scores keep id order
  });
  for (int32_t s = 0; s < S; ++s) {
    int32_t* o = out + (size_t)s * m;
    if (s == 0) {
      std::copy(base.begin(), base.end(), o);
    } else if (s == 1) {
      std::reverse_copy(base.begin(), base.end(), o);
    } else {
      uint64_t st = seed + (uint64_t)s;
      for (int32_t h = 0; h < m; ++h) o[h] = h;
      for (int32_t i = m - 1; i >= 1; --i) {
        const int32_t j = (int32_t)(splitmix64_next(st) % (uint64_t)(i + 1));
        std::swap(o[i], o[j]);
      }
    }
  }
}

// ------------------------------------------------------------ context ---

int env_int(const char* name, int dflt) {
  const char* v = std::getenv(name);
  return (v && *v) ? std::atoi(v) : dflt;
}

}  // namespace

struct pp_ctx {
  int device = 0;
  hipStream_t own = nullptr;
  // problem, preorder layout
  DevBuf lam, w, f, meta;
  // tree tables in one allocation (one upload): next positions, preorder
  // (position -> caller id) and the backtrack's skip-chain table
  DevBuf tree;
  int32_t* nextpos = nullptr;
  int32_t* order = nullptr;
  uint32_t* ce = nullptr;
  // uploads for host-pointer entry points (caller order)
  DevBuf up_lam, up_w, up_f, up_u8;
  // per-slot state
  DevBuf tgt, v1, v2, h1, profit, sel, bits, ring, cs;
  DevBuf sel0;  // standalone selections, [m][npad/32] (greedy position 0)
  DevBuf partial, flag, gx, gxp;
  DevBuf sp_lists, spill;  // spilled skip rows of deep trees
  uint32_t epoch = 0;
  std::vector<uint32_t> meta_host;  // source of the last metadata upload
  std::vector<uint8_t> tree_host;   // and of the last tree tables
  std::vector<hipEvent_t> events;
  // pinned host copy of the chain states read back after each refinement
  // launch (a direct device-to-host copy)
  ChainState* cs_pin = nullptr;
  size_t cs_pin_n = 0;
  uint64_t* val_pin = nullptr;  // pinned read-back of the input checks
  // pinned staging of the tree tables uploaded per call (copies from
  // pageable memory would each wait for the stream); filled front to back
  // and reused once the copies out of it have completed: stage_ev is
  // recorded on stage_st after the latest copy, and every earlier copy not
  // known to be complete is on that stream too
  uint8_t* stage = nullptr;
  size_t stage_cap = 0, stage_used = 0;
  hipEvent_t stage_ev = nullptr;
  hipStream_t stage_st = nullptr;
  bool stage_pending = false;
  ~pp_ctx() {
    if (cs_pin) (void)hipHostFree(cs_pin);
    if (stage) (void)hipHostFree(stage);
    if (stage_ev) (void)hipEventDestroy(stage_ev);
    if (val_pin) (void)hipHostFree(val_pin);
    for (DevBuf* b : {&lam, &w, &f, &tree, &meta, &up_lam, &up_w,
                      &up_f, &up_u8, &tgt, &v1, &v2, &h1, &profit, &sel, &sel0, &bits,
                      &ring, &cs, &partial, &flag, &gx, &gxp, &sp_lists, &spill})
      b->release();
    for (hipEvent_t e : events) (void)hipEventDestroy(e);
    if (own) (void)hipStreamDestroy(own);
  }
};

namespace {

int select_device(pp_ctx* c) {
  PP_HIP(hipSetDevice(c->device));
  return PP_OK;
}

// At least `count` pinned chain states in c->cs_pin.
int ensure_cs_pin(pp_ctx* c, size_t count) {
  if (c->cs_pin_n >= count) return PP_OK;
  if (c->cs_pin) PP_HIP(hipHostFree(c->cs_pin));
  c->cs_pin = nullptr;
  c->cs_pin_n = 0;
  PP_HIP(hipHostMalloc((void**)&c->cs_pin, count * sizeof(ChainState), hipHostMallocDefault));
  c->cs_pin_n = count;
  return PP_OK;
}

int ensure_val_pin(pp_ctx* c) {
  if (!c->val_pin)
    PP_HIP(hipHostMalloc((void**)&c->val_pin, 2 * kValidateBlocks * sizeof(uint64_t),
                         hipHostMallocDefault));
  return PP_OK;
}

// Host-to-device copy of `bytes` at `src` (which the caller may reuse at
// once) through the context's pinned staging buffer.
int stage_h2d(pp_ctx* c, void* dst, const void* src, size_t bytes, hipStream_t st) {
  if (bytes == 0) return PP_OK;
  const size_t need = (bytes + 255) & ~(size_t)255;
  // copies on another stream, or a full buffer: wait for the copies out of
  // it, then fill it from the front
  if (c->stage_pending && (c->stage_st != st || c->stage_used + need > c->stage_cap)) {
    PP_HIP(hipEventSynchronize(c->stage_ev));
    c->stage_pending = false;
    c->stage_used = 0;
  }
  if (c->stage_used + need > c->stage_cap) {
    c->stage_used = 0;
    if (need > c->stage_cap) {
      const size_t cap = std::max({need * 4, c->stage_cap * 2, (size_t)1 << 20});
      if (c->stage) PP_HIP(hipHostFree(c->stage));
      c->stage = nullptr;
      c->stage_cap = 0;
      PP_HIP(hipHostMalloc((void**)&c->stage, cap, hipHostMallocDefault));
      c->stage_cap = cap;
    }
  }
  std::memcpy(c->stage + c->stage_used, src, bytes);
  PP_HIP(hipMemcpyAsync(dst, c->stage + c->stage_used, bytes, hipMemcpyHostToDevice, st));
  c->stage_used += need;
  if (!c->stage_ev) PP_HIP(hipEventCreateWithFlags(&c->stage_ev, hipEventDisableTiming));
  PP_HIP(hipEventRecord(c->stage_ev, st));
  c->stage_st = st;
  c->stage_pending = true;
  return PP_OK;
}

// Waits for `st` by polling (every wait of the library): the host decides
// the next launches from what it reads back (after each refinement launch,
// the chain states), so the wake-up delay of a blocking wait would leave
// the device idle, and for small trees it is a large part of a call.
int poll_stream(hipStream_t st) {
  for (;;) {
    const hipError_t q = hipStreamQuery(st);
    if (q == hipSuccess) return PP_OK;
    if (q != hipErrorNotReady) PP_HIP(q);
  }
}

int npad_of(int32_t n) { return (n + 63) / 64 * 64; }

// Allocate per-slot buffers for `slots` chains of up to `kmax` cells.
int ensure_slots(pp_ctx* c, DevState& d, int32_t slots, int32_t kmax,
                 int cells) {
  const size_t n = (size_t)d.n, m = (size_t)d.m, npad = (size_t)d.npad;
  const int32_t stages = std::max(1, (kmax + 64 * cells - 1) / (64 * cells));
  PP_TRY(c->tgt.ensure(slots * m * n));
  PP_TRY(c->v1.ensure(slots * m * n * 8));
  PP_TRY(c->v2.ensure(slots * m * n * 8));
  PP_TRY(c->h1.ensure(slots * m * n));
  PP_TRY(c->profit.ensure(slots * n * 8));
  PP_TRY(c->sel.ensure(slots * (npad / 8)));
  PP_TRY(c->bits.ensure((size_t)slots * stages * cells * npad * 8));
  // ring words carry a launch tag; fresh memory is zeroed so that no stale
  // word can ever carry a live tag (tags start at 1)
  PP_TRY(c->ring.ensure((size_t)slots * stages * npad * 16, true));
  PP_TRY(c->cs.ensure(slots * sizeof(ChainState)));
  d.tgt = c->tgt.as<uint8_t>();
  d.v1 = c->v1.as<int64_t>();
  d.v2 = c->v2.as<int64_t>();
  d.h1 = c->h1.as<uint8_t>();
  d.profit = c->profit.as<int64_t>();
  d.sel = c->sel.as<uint32_t>();
  d.bits = c->bits.as<uint64_t>();
  d.ring = c->ring.as<uint64_t>();
  d.cs = c->cs.as<ChainState>();
  d.stages = stages;
  d.cells = cells;
  return PP_OK;
}

// Real-valued costs: exact objective values per slot and the per-block
// partials of one launch of up to kMaxChains chains.
int ensure_exact(pp_ctx* c, DevState& d, int32_t slots) {
  d.gx_blocks = gexact_blocks(d.n, d.m);
  PP_TRY(c->gx.ensure((size_t)slots * 2 * kExLimbs * 4));
  PP_TRY(c->gxp.ensure((size_t)kMaxChains * d.gx_blocks * kExLimbs * 8));
  d.gx = c->gx.as<uint32_t>();
  d.gxp = c->gxp.as<uint64_t>();
  return PP_OK;
}

// Exact objective values of `count` consecutive slots from `first`.
int read_exact(const DevState& d, int32_t first, int32_t count, hipStream_t st,
               std::vector<uint32_t>& out) {
  // slot s's G is gx[2s]: one copy of the slots' pairs, then every other
  std::vector<uint32_t> pairs((size_t)count * 2 * kExLimbs);
  PP_HIP(hipMemcpyAsync(pairs.data(), d.gx + (size_t)first * 2 * kExLimbs,
                        pairs.size() * sizeof(uint32_t), hipMemcpyDeviceToHost, st));
  PP_TRY(poll_stream(st));
  out.assign((size_t)count * kExLimbs, 0);
  for (int32_t q = 0; q < count; ++q)
    std::memcpy(out.data() + (size_t)q * kExLimbs, pairs.data() + (size_t)q * 2 * kExLimbs,
                kExLimbs * sizeof(uint32_t));
  return PP_OK;
}

ChainSet chain_set(const std::vector<int32_t>& slots,
                   const std::vector<int32_t>& workers,
                   const std::vector<int32_t>& kprime, size_t lo, size_t hi) {
  ChainSet s;
  std::memset(&s, 0, sizeof s);
  s.count = (int32_t)(hi - lo);
  for (size_t k = lo; k < hi; ++k) {
    s.slot[k - lo] = slots[k];
    s.src[k - lo] = slots[k];
    s.worker[k - lo] = workers[k];
    s.kprime[k - lo] = kprime[k];
  }
  return s;
}

struct Timer {
  bool on = false;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> marks;
  size_t used = 0;
};

int timer_mark(pp_ctx* c, Timer& t, bool start, hipStream_t st) {
  if (!t.on) return PP_OK;
  if (start) {
    while (c->events.size() < 2 * (t.used + 1)) {
      hipEvent_t e;
      PP_HIP(hipEventCreate(&e));
      c->events.push_back(e);
    }
    t.marks.push_back({c->events[2 * t.used], c->events[2 * t.used + 1]});
    PP_HIP(hipEventRecord(t.marks.back().first, st));
  } else {
    PP_HIP(hipEventRecord(t.marks.back().second, st));
    ++t.used;
  }
  return PP_OK;
}

struct Engine {
  pp_ctx* c;
  DevState d;
  int32_t slots_lds;
  int resident;       // DP blocks resident at once
  uint32_t spin_limit;
  int fmax = 0;  // every DP value < 2^62: max via v_max_f64
  hipStream_t st;
  Timer timer;

  // One DP sweep over the chains of `set` (kprime >= 1 each), split into
  // launches whose stages all fit on the device at once.
  int dp(const ChainSet& in, int store_bits) {
    if (!d.meta || !d.profit || !d.bits || !d.ring || !d.cs)
      return fail(PP_E_DEVICE, "internal: DP sweep buffers are not set");
    const int cellsw = 64 * d.cells;
    int32_t k = 0;
    while (k < in.count) {
      ChainSet s;
      std::memset(&s, 0, sizeof s);
      int32_t blocks = 0;
      while (k < in.count) {
        const int32_t g = (in.kprime[k] + cellsw - 1) / cellsw;
        if (s.count > 0 && blocks + g > resident) break;
        s.slot[s.count] = in.slot[k];
        s.src[s.count] = in.src[k];
        s.worker[s.count] = in.worker[k];
        s.kprime[s.count] = in.kprime[k];
        s.base[s.count] = blocks;
        blocks += g;
        ++s.count;
        ++k;
      }
      s.base[s.count] = blocks;
      if (blocks > resident)
        return fail(PP_E_UNSUPPORTED,
                    "capacity needs more DP stages than the device holds");
      if (++c->epoch == 0) ++c->epoch;  // tag 0 marks never-written words
      PP_TRY(timer_mark(c, timer, true, st));
      PP_HIP(launch_dp(s, d, c->epoch, spin_limit, store_bits, slots_lds, fmax,
                       st));
      PP_TRY(timer_mark(c, timer, false, st));
    }
    return PP_OK;
  }

  // Greedy position 0 of every chain of `set`: the standalone solve of its
  // worker (its selection saved in sel0), adopted and committed.
  int take_standalone(const ChainSet& set, const uint32_t* sel0) {
    if (set.count == 0) return PP_OK;
    PP_HIP(launch_take_standalone(set, d, sel0, st));
    if (d.f64) PP_HIP(launch_gexact(set, d, kModeGreedy, st));  // exact G, marks
    PP_HIP(launch_commit(set, d, kModeGreedy, st));
    return PP_OK;
  }

  // One worker update (gains, DP sweep, accept + backtrack, commit) for
  // every chain of `set`.
  int update(const ChainSet& set, int mode) {
    if (set.count == 0) return PP_OK;
    PP_HIP(launch_gains(set, d, st, kGainsMarginal, mode == kModeRefine ? 1 : 0));
    PP_TRY(dp(set, 1));
    PP_HIP(launch_backtrack(set, d, mode, st));
    if (d.f64) PP_HIP(launch_gexact(set, d, mode, st));  // exact G and the decision
    PP_HIP(launch_commit(set, d, mode, st));
    return PP_OK;
  }
};

// Cells per lane for a launch whose chains need `total_stage_cells_c1`
// stages at one cell per lane.  A stage's compute wave, alone on its SIMD,
// takes about 37 ns per row step at one cell per lane (bound by the wave's
// instruction issue); the weights below (45 / 61 / 96 at 1 / 2 / 4 cells
// per lane) are relative row-step costs of the sweep at each width.  When
// compute waves outnumber SIMDs they share the SIMDs' vector units, so the
// estimate is scaled by the waves per SIMD (about three quarters of a
// step's instructions are vector ops).
// Only widths whose stages all fit on the device at once are considered; if
// none fits, the width with the most resident blocks is used and launches
// are split.
int choose_cells(int32_t total_stage_cells_c1, int dev, int32_t slots_lds) {
  const int forced = env_int("PP_DP_CELLS", 0);
  if (forced == 1 || forced == 2 || forced == 4) return forced;
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    cus = 256;
  const double simds = 4.0 * cus;
  const struct { int c; double ns; } widths[] = {{1, 45.0}, {2, 61.0}, {4, 96.0}};
  int best = 0, most = 2, most_res = 0;
  double best_cost = 0.0;
  for (const auto& w : widths) {
    const int res = dp_resident_blocks(w.c, slots_lds, dev);
    const int32_t stages = (total_stage_cells_c1 + w.c - 1) / w.c;
    if (res > most_res) {
      most = w.c;
      most_res = res;
    }
    if (res <= 0 || stages > res) continue;
    const double cost = w.ns * std::max(1.0, 0.75 * stages / simds);
    if (best == 0 || cost < best_cost) {
      best = w.c;
      best_cost = cost;
    }
  }
  return best ? best : most;
}

struct PlanResult {
  std::vector<int64_t> start_obj, standalone;
  std::vector<int32_t> sweeps, accepts, orders;
  int32_t best = 0, S = 0;     // best: start index, or S + c for safeguard c
  int32_t win_slot = 0;        // slot holding the returned placement
  int64_t win_obj = 0;         // its objective
  bool sg_run = false;         // safeguard candidates evaluated
  int64_t sg_obj[3] = {0, 0, 0};
  int32_t extra_slot = -1;     // first slot reserved for the caller
  int64_t skipped_cells = 0;   // cells of updates resolved without a sweep
  int64_t spec_cells = 0;      // cells swept by discarded speculative updates
  int64_t updates = 0, cells = 0;
  double dp_ms = 0.0;
  int32_t dp_launches = 0;
  int32_t restarts = 0;        // plan runs repeated after a DP sweep stalled
  int32_t lane_cells = 0;      // DP cells per lane of the sweep
  int32_t fmax = 0;            // maximum by one 64-bit float instruction
  // real-valued costs: exact objective values of the starts and of the
  // returned placement (kExLimbs limbs each)
  std::vector<uint32_t> start_gx, win_gx;
};

// Comparator safeguards of Sec. IV-C (Algorithm 1: the candidate set also
// holds the Independent, Popularity and LocalDedup placements when costs are
// requester-side).  Independent and Popularity solve every worker's DP as
// concurrent chains in scratch slots 0..m-1 and assemble the selections into
// their candidate slot; LocalDedup runs the workers in increasing id, each
// against the union of the earlier ones, in its own slot.  A candidate is
// returned only if strictly better than the best start; Independent,
// Popularity, LocalDedup break ties in that order.
int run_safeguards(Engine& e, int32_t m, const std::vector<int32_t>& kp,
                   int32_t slot_b, int64_t cells_pass, hipStream_t st,
                   PlanResult& res) {
  pp_ctx* c = e.c;
  DevState& d = e.d;
  const size_t mn = (size_t)m * d.n;
  PP_TRY(c->flag.ensure(64));
  PP_HIP(hipMemsetAsync(c->flag.p, 0, 4, st));
  PP_HIP(launch_requester_check(d.f, d.n, m, c->flag.as<int32_t>(), st));
  int32_t mismatch = 0;
  PP_HIP(hipMemcpyAsync(&mismatch, c->flag.p, 4, hipMemcpyDeviceToHost, st));
  PP_TRY(poll_stream(st));
  if (mismatch) return PP_OK;  // source-dependent costs: no comparators
  // keep the best start's placement out of the scratch slots
  PP_HIP(hipMemcpyAsync(d.tgt + (size_t)slot_b * mn, d.tgt + (size_t)res.win_slot * mn,
                        mn, hipMemcpyDeviceToDevice, st));
  if (d.f64)
    PP_HIP(hipMemcpyAsync(d.gx + (size_t)slot_b * 2 * kExLimbs,
                          d.gx + (size_t)res.win_slot * 2 * kExLimbs, 2 * kExLimbs * 4,
                          hipMemcpyDeviceToDevice, st));
  res.win_slot = slot_b;
  std::vector<int32_t> cand_slot = {slot_b + 1, slot_b + 2, slot_b + 3};
  {
    std::vector<int32_t> z(3, 0);
    PP_HIP(launch_init_slots(chain_set(cand_slot, z, z, 0, 3), d, 1, st));
  }
  // Independent and Popularity: every worker's DP at once
  std::vector<int32_t> sl, wk, kk;
  for (int32_t h = 0; h < m; ++h)
    if (kp[h] > 0) {
      sl.push_back(h);
      wk.push_back(h);
      kk.push_back(kp[h]);
    }
  const int gm[2] = {kGainsIndependent, kGainsPopularity};
  for (int q = 0; q < 2; ++q) {
    for (size_t lo = 0; lo < sl.size(); lo += kMaxChains) {
      const size_t hi = std::min(sl.size(), lo + (size_t)kMaxChains);
      const ChainSet set = chain_set(sl, wk, kk, lo, hi);
      PP_HIP(launch_init_slots(set, d, 0, st));
      PP_HIP(launch_gains(set, d, st, gm[q]));
      PP_TRY(e.dp(set, 1));
      PP_HIP(launch_backtrack(set, d, kModeGreedy, st));
      PP_HIP(launch_assemble(set, d, cand_slot[q], st));
    }
  }
  {
    std::vector<int32_t> z(2, 0), two(cand_slot.begin(), cand_slot.begin() + 2);
    PP_HIP(launch_holder_build(chain_set(two, z, z, 0, 2), d, st));
  }
  // LocalDedup: workers in increasing id, each one update in slot B+3
  for (int32_t h = 0; h < m; ++h) {
    if (kp[h] == 0) continue;
    const std::vector<int32_t> s1 = {cand_slot[2]}, w1 = {h}, k1 = {kp[h]};
    const ChainSet set = chain_set(s1, w1, k1, 0, 1);
    PP_HIP(launch_gains(set, d, st, kGainsLocalDedup));
    PP_TRY(e.dp(set, 1));
    PP_HIP(launch_backtrack(set, d, kModeGreedy, st));
    if (d.f64) PP_HIP(launch_gexact(set, d, kModeGreedy, st));  // adopts T'_h
    PP_HIP(launch_commit(set, d, kModeGreedy, st));
  }
  {
    std::vector<int32_t> z(3, 0);
    PP_HIP(launch_objective(chain_set(cand_slot, z, z, 0, 3), d, st));
  }
  std::vector<ChainState> fin(3);
  PP_HIP(hipMemcpyAsync(fin.data(), d.cs + cand_slot[0], sizeof(ChainState) * 3,
                        hipMemcpyDeviceToHost, st));
  PP_TRY(poll_stream(st));
  // the scratch chains' status words, in case a DP wait gave up
  std::vector<ChainState> scr(m);
  PP_HIP(hipMemcpyAsync(scr.data(), d.cs, sizeof(ChainState) * m,
                        hipMemcpyDeviceToHost, st));
  PP_TRY(poll_stream(st));
  for (const ChainState& x : fin)
    if (x.status) return stall_fail();
  for (const ChainState& x : scr)
    if (x.status) return stall_fail();
  res.sg_run = true;
  std::vector<uint32_t> cgx;
  if (d.f64) PP_TRY(read_exact(d, cand_slot[0], 3, st, cgx));
  for (int q = 0; q < 3; ++q) {
    res.sg_obj[q] = fin[q].obj;
    // real-valued costs compare exact values
    const bool better = d.f64 ? ex_cmp(&cgx[(size_t)q * kExLimbs], res.win_gx.data()) > 0
                              : fin[q].obj > res.win_obj;
    if (better) {
      res.win_obj = fin[q].obj;
      res.win_slot = cand_slot[q];
      res.best = res.S + q;
      if (d.f64) res.win_gx.assign(cgx.begin() + (size_t)q * kExLimbs,
                                   cgx.begin() + (size_t)(q + 1) * kExLimbs);
    }
  }
  res.updates += 3 * (int64_t)m;
  res.cells += 3 * cells_pass;
  return PP_OK;
}

// Coordinate refinement (Algorithm 1's sweeps) of the starts `starts`,
// after their greedy pass.  Each start keeps its own position and sweep.
// The host mirrors every start's stale-input marks (ChainState::dirty, the
// same rules as the kernels: a worker's sweep clears its bit, an adopted
// replacement sets every other worker's) and passes over positions whose
// update is resolved as rejected without a sweep (a clean worker, or
// k = 0) at no cost.  Each launch then holds every active start's next
// update that needs a sweep, in the start's own slot, and fills the rest of
// `budget` with speculative updates: later positions of the same sweep of
// a start, in spare slots, computed against the start's current placement,
// which is the placement each of them sees in Algorithm 1's order as long
// as every earlier one is rejected.  The first accepted update of a start
// is adopted and committed; the positions after it are looked at again in
// the next launch.  A start whose sweep has accepted an update goes on into
// its next sweep the same way once the rest of the sweep is in the launch.
// Results are those of the sequential sweeps.
int refine_starts(Engine& e, const std::vector<int32_t>& starts, int32_t spare_base,
                  int32_t budget, int32_t block_budget, int32_t m,
                  const std::vector<int32_t>& kp, int32_t max_rounds, PlanResult& res) {
  DevState& d = e.d;
  const int32_t A = (int32_t)starts.size();
  for (int32_t q = 1; q < A; ++q)
    if (starts[q] != starts[0] + q) return fail(PP_E_DEVICE, "internal: start slots");
  struct St {
    int32_t s, pos;
    bool improved, done;
    uint32_t dirty[8];
    bool is_dirty(int32_t h) const { return (dirty[h >> 5] >> (h & 31)) & 1u; }
    void mark_ran(int32_t h) { dirty[h >> 5] &= ~(1u << (h & 31)); }
    void mark_adopted(int32_t h) {
      for (int q = 0; q < 8; ++q) dirty[q] = ~0u;
      mark_ran(h);
    }
  };
  std::vector<St> st(A);
  {
    std::vector<ChainState> cs0(A);
    PP_HIP(hipMemcpyAsync(cs0.data(), d.cs + starts[0], sizeof(ChainState) * A,
                          hipMemcpyDeviceToHost, e.st));
    PP_TRY(poll_stream(e.st));
    for (int32_t q = 0; q < A; ++q) {
      if (cs0[q].status) return stall_fail();
      st[q].s = starts[q];
      st[q].pos = 0;
      st[q].improved = false;
      st[q].done = false;
      std::memcpy(st[q].dirty, cs0[q].dirty, sizeof st[q].dirty);
    }
  }
  auto worker_at = [&](const St& x, int32_t a) { return res.orders[(size_t)x.s * m + a]; };
  auto resolved_free = [&](const St& x, int32_t a) {
    const int32_t h = worker_at(x, a);
    return kp[h] == 0 || !x.is_dirty(h);
  };
  auto free_cells = [&](const St& x, int32_t a) {
    return (int64_t)d.n * kp[worker_at(x, a)];  // 0 for k = 0
  };
  struct Item {
    int32_t q, slot, worker, pos;
    bool next;  // a position of the start's next sweep
  };
  for (;;) {
    // each start's next update that needs a sweep; sweep ends
    for (int32_t q = 0; q < A; ++q) {
      St& x = st[q];
      while (!x.done) {
        if (x.pos == m) {
          res.sweeps[x.s] += 1;
          const bool improved = x.improved;
          const bool capped = max_rounds > 0 && res.sweeps[x.s] >= max_rounds;
          if (!improved || capped) {
            x.done = true;
            break;
          }
          x.pos = 0;
          x.improved = false;
          continue;
        }
        if (!resolved_free(x, x.pos)) break;
        res.skipped_cells += free_cells(x, x.pos);
        ++x.pos;
      }
    }
    std::vector<Item> items;
    std::vector<int32_t> scan(A, m), wscan(A, 0);
    // A start whose sweep has accepted a replacement sweeps again unless the
    // cap stops it, so once every later position of this sweep is in the
    // launch or resolved without a sweep, positions of the next sweep can be
    // speculated too (valid if everything before them is rejected).
    std::vector<char> can_wrap(A, 0);
    for (int32_t q = 0; q < A; ++q)
      if (!st[q].done) {
        items.push_back({q, st[q].s, worker_at(st[q], st[q].pos), st[q].pos, false});
        scan[q] = st[q].pos + 1;
        can_wrap[q] = st[q].improved && (max_rounds == 0 || res.sweeps[st[q].s] + 1 < max_rounds);
      }
    if (items.empty()) return PP_OK;
    // speculative updates: at most `budget` updates in all (one spare slot
    // each; budget - 1 spare slots exist) and, beyond the starts' own
    // updates, at most `block_budget` DP stage blocks in the launch
    const int32_t cellsw = 64 * d.cells;
    auto blocks_of = [&](int32_t h) { return (kp[h] + cellsw - 1) / cellsw; };
    int32_t blocks = 0;
    for (const Item& it : items) blocks += blocks_of(it.worker);
    int32_t spares = 0;
    auto room = [&]() { return (int32_t)items.size() < budget && spares < budget - 1; };
    // a position b < pos of the next sweep needs a sweep there (if nothing
    // is adopted before it) iff its worker is stale now: the workers of
    // positions >= pos run in this launch or are unchanged since their last
    // sweep
    auto next_needs_sweep = [&](const St& x, int32_t b) {
      const int32_t h = worker_at(x, b);
      return kp[h] > 0 && x.is_dirty(h);
    };
    for (bool grew = true; grew && room();) {
      grew = false;
      for (int32_t q = 0; q < A && room(); ++q) {
        if (st[q].done) continue;
        int32_t a = scan[q];
        while (a < m && resolved_free(st[q], a)) ++a;
        if (a < m && blocks + blocks_of(worker_at(st[q], a)) > block_budget) {
          scan[q] = m;  // this start's next update does not fit any more
          can_wrap[q] = 0;
          continue;
        }
        if (a < m) {
          blocks += blocks_of(worker_at(st[q], a));
          items.push_back({q, spare_base + spares++, worker_at(st[q], a), a, false});
          scan[q] = a + 1;
          grew = true;
          continue;
        }
        scan[q] = m;
        if (!can_wrap[q]) continue;
        int32_t b = wscan[q];
        while (b < st[q].pos && !next_needs_sweep(st[q], b)) ++b;
        if (b >= st[q].pos || blocks + blocks_of(worker_at(st[q], b)) > block_budget) {
          can_wrap[q] = 0;
          continue;
        }
        blocks += blocks_of(worker_at(st[q], b));
        items.push_back({q, spare_base + spares++, worker_at(st[q], b), b, true});
        wscan[q] = b + 1;
        grew = true;
      }
    }
    std::stable_sort(items.begin(), items.end(),
                     [](const Item& u, const Item& v) { return u.q < v.q; });
    ChainSet set;
    std::memset(&set, 0, sizeof set);
    set.count = (int32_t)items.size();
    for (int32_t k = 0; k < set.count; ++k) {
      set.slot[k] = items[k].slot;
      set.src[k] = st[items[k].q].s;
      set.worker[k] = items[k].worker;
      set.kprime[k] = kp[items[k].worker];
    }
    PP_HIP(launch_gains(set, d, e.st, kGainsMarginal, 1));
    PP_TRY(e.dp(set, 1));
    PP_HIP(launch_backtrack(set, d, kModeRefine, e.st));
    if (d.f64) PP_HIP(launch_gexact(set, d, kModeRefine, e.st));
    // the launch's results, to pinned memory in one copy: the starts' slots
    // (consecutive) through the last spare slot used (the slots between
    // them come along unread)
    const size_t span = spares > 0 ? (size_t)(spare_base + spares - starts[0]) : (size_t)A;
    PP_TRY(ensure_cs_pin(e.c, span));
    ChainState* own = e.c->cs_pin;
    ChainState* spare = e.c->cs_pin + (spare_base - starts[0]);
    PP_HIP(hipMemcpyAsync(own, d.cs + starts[0], sizeof(ChainState) * span,
                          hipMemcpyDeviceToHost, e.st));
    PP_TRY(poll_stream(e.st));
    std::vector<ChainState> cs(items.size());
    for (size_t k = 0; k < items.size(); ++k)
      cs[k] = items[k].slot >= spare_base ? spare[items[k].slot - spare_base]
                                          : own[items[k].slot - starts[0]];
    // decisions, in each start's order
    std::vector<int32_t> csl, cwk, ckp;
    AdoptSet ad;
    ad.count = 0;
    size_t k = 0;
    for (int32_t q = 0; q < A; ++q) {
      St& x = st[q];
      uint32_t ran[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      const Item* take = nullptr;
      int32_t last = x.pos - 1;  // last position resolved in this launch
      bool in_next = false;
      for (; k < items.size() && items[k].q == q; ++k) {
        const Item& it = items[k];
        const ChainState& c = cs[k];
        if (c.status) return stall_fail();
        if (take) {  // computed against a placement that has changed
          if (!c.skip) res.spec_cells += (int64_t)d.n * kp[it.worker];
          continue;
        }
        if (it.next && !in_next) {
          // every position left in this sweep was rejected: the sweep ends
          // (it accepted earlier, so the next one follows)
          for (int32_t a = last + 1; a < m; ++a) res.skipped_cells += free_cells(x, a);
          res.sweeps[x.s] += 1;
          x.improved = false;
          last = -1;
          in_next = true;
        }
        // positions passed over on the way are resolved as rejected
        for (int32_t a = last + 1; a < it.pos; ++a) res.skipped_cells += free_cells(x, a);
        if (c.skip) res.skipped_cells += (int64_t)d.n * kp[it.worker];
        last = it.pos;
        if (c.accept) {
          take = &it;
          x.improved = true;
          x.mark_adopted(it.worker);
        } else {
          x.mark_ran(it.worker);
          if (it.slot != x.s) ran[it.worker >> 5] |= 1u << (it.worker & 31);
        }
      }
      if (x.done) continue;
      x.pos = last + 1;
      bool any_ran = false;
      for (uint32_t b : ran) any_ran = any_ran || b != 0;
      // (an update in the start's own slot is backtracked and marked by
      // k_backtrack itself)
      if ((take && take->slot != x.s) || (!take && any_ran)) {
        const int32_t q2 = ad.count++;
        ad.slot[q2] = x.s;
        ad.from[q2] = take ? take->slot : -1;
        ad.worker[q2] = take ? take->worker : 0;
        std::memcpy(ad.ran[q2], ran, sizeof ran);
      }
      if (take) {
        csl.push_back(x.s);
        cwk.push_back(take->worker);
        ckp.push_back(kp[take->worker]);
      }
    }
    PP_HIP(launch_adopt(ad, d, e.st));
    if (!csl.empty())
      PP_HIP(launch_commit(chain_set(csl, cwk, ckp, 0, csl.size()), d, kModeRefine, e.st));
  }
}

int run_plan_once(pp_ctx* c, const TreeLayout& t, int32_t m, const int32_t* cap,
                  const pp_options& o, bool fmax_ok, hipStream_t st, PlanResult& res,
                  int32_t extra_slots, bool f64, double eps, int attempt);

// Algorithm 1 on the context's inputs, run again (identical results: the
// plan is deterministic) if a DP sweep stalled.
int run_plan(pp_ctx* c, const TreeLayout& t, int32_t m, const int32_t* cap,
             const pp_options& o, bool fmax_ok, hipStream_t st,
             PlanResult& res, int32_t extra_slots = 0, bool f64 = false,
             double eps = 0.0) {
  for (int attempt = 0;; ++attempt) {
    g_stall = false;
    res = PlanResult{};
    const int rc = run_plan_once(c, t, m, cap, o, fmax_ok, st, res, extra_slots, f64, eps,
                                 attempt);
    res.restarts = attempt;
    if (rc == PP_OK || !g_stall || attempt >= kStallRetries) return rc;
    PP_TRY(poll_stream(st));
  }
}

// Spin limit of the DP sweep's bounded waits: PP_SPIN_LIMIT (a test hook)
// on the first attempt, then at least the default, four times longer per
// further attempt.
uint32_t spin_limit_for(int attempt) {
  const uint32_t base = (uint32_t)env_int("PP_SPIN_LIMIT", (int)kDefaultSpin);
  if (attempt == 0) return base;
  uint64_t v = std::max(base, kDefaultSpin);
  for (int a = 1; a < attempt; ++a) v *= 4;
  return (uint32_t)std::min<uint64_t>(v, 1u << 30);
}

// Algorithm 1 on device-resident, preorder-laid-out inputs in `c`.
// Real-valued costs (f64): every value is the bit pattern of a non-negative
// double, so the comparisons below (orders, best start) hold unchanged.
int run_plan_once(pp_ctx* c, const TreeLayout& t, int32_t m, const int32_t* cap,
                  const pp_options& o, bool fmax_ok, hipStream_t st, PlanResult& res,
                  int32_t extra_slots, bool f64, double eps, int attempt) {
  const int32_t n = t.n;
  const int32_t S = num_starts(m, o.n_starts);
  res.S = S;
  std::vector<int32_t> kp(m);
  int32_t kmax = 0;
  int64_t cells_pass = 0;
  for (int32_t h = 0; h < m; ++h) {
    kp[h] = std::min(cap[h], n);
    kmax = std::max(kmax, kp[h]);
    cells_pass += (int64_t)n * kp[h];
  }
  // safeguards (requester-side inputs only): after the starts, slot B keeps
  // the best start's placement, slots B+1..B+3 the Independent, Popularity
  // and LocalDedup candidates, and slots 0..m-1 serve as scratch chains
  const bool sg_asked = (o.flags & PP_F_SAFEGUARDS) != 0;
  const int32_t slot_b = std::max(m, S);
  // stage blocks a speculative launch may fill: three per compute unit (the
  // sweep gives each block's compute wave a SIMD of its own where the
  // placement allows; a fourth block per unit slows every stage on it), and
  // never more than fit the device at once
  int32_t spec_blocks = 768;
  {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, c->device) ==
            hipSuccess && cus > 0)
      spec_blocks = 3 * cus;
    spec_blocks = env_int("PP_SPEC_BLOCKS", spec_blocks);
  }
  // speculative refinement: up to kSpecChains updates per launch (each
  // start's next one and later positions of the same sweep, all but the
  // first of a start in spare slots at the end); twice as many where that
  // many chains of the widest capacity (stages at one cell per lane) fit
  // the launch's stage blocks -- small capacities, whose launches take the
  // same time with more chains
  const int32_t wide_stages = std::max(1, (kmax + 63) / 64);
  const int32_t spec_default =
      2 * kSpecChains * wide_stages <= spec_blocks ? 2 * kSpecChains : kSpecChains;
  const int32_t spec_chains =  // updates per refinement launch
      env_int("PP_NO_SPEC", 0) ? 1
                               : std::max(1, std::min(kMaxChains, env_int("PP_SPEC_CHAINS",
                                                                          spec_default)));
  const int32_t spare_base = slot_b + (sg_asked ? 4 : 0) + extra_slots;
  const int32_t slots = spare_base + (spec_chains > 1 ? spec_chains - 1 : 0);
  res.extra_slot = extra_slots > 0 ? slot_b + (sg_asked ? 4 : 0) : -1;
  Engine e;
  e.c = c;
  e.st = st;
  e.slots_lds = t.slots;
  e.spin_limit = spin_limit_for(attempt);
  e.timer.on = (o.flags & PP_F_TIME_KERNELS) != 0;
  DevState& d = e.d;
  d = DevState{};
  d.n = n;
  d.m = m;
  d.npad = npad_of(n);
  d.lam = c->lam.as<int64_t>();
  d.w = c->w.as<int64_t>();
  d.f = c->f.as<int64_t>();
  d.nextpos = c->nextpos;
  d.ce = c->ce;
  // widest single launch: every start's update at once
  int64_t stage64 = 0;
  {
    std::vector<int32_t> ks(kp.begin(), kp.end());
    std::sort(ks.rbegin(), ks.rend());
    for (int32_t k = 0; k < std::min<int32_t>(S, kMaxChains); ++k)
      stage64 += (ks[k % m] + 63) / 64;
  }
  const int cells = choose_cells((int32_t)std::min<int64_t>(stage64, INT32_MAX),
                                 c->device, e.slots_lds);
  {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, c->device) ==
            hipSuccess && cus > 0)
      d.role_max_blocks = 4 * cus;
  }
  e.resident = dp_resident_blocks(cells, e.slots_lds, c->device);
  if (attempt > 0 && e.resident > 0) {
    // fewer stage blocks per launch, but every chain's stages in one
    const int32_t chain = (kmax + 64 * cells - 1) / (64 * cells);
    e.resident = std::max(chain, e.resident >> attempt);
  }
  if (e.resident <= 0)
    return fail(PP_E_UNSUPPORTED, "DP sweep cannot be resident (LDS stack of " +
                                      std::to_string(e.slots_lds) + " rows)");
  e.fmax = fmax_ok && env_int("PP_DP_NO_FMAX", 0) == 0;
  res.lane_cells = cells;
  res.fmax = (e.fmax || f64) ? 1 : 0;
  PP_TRY(ensure_slots(c, d, slots, kmax, cells));
  if (f64) {
    d.f64 = 1;
    d.eps = eps;
    PP_TRY(ensure_exact(c, d, slots));
  }
  PP_TRY(upload_meta(c, t, cells, st));
  d.meta = c->meta.as<uint32_t>();  // upload_meta may have (re)allocated it
  PP_TRY(upload_spills(c, t, d, slots, st));

  // --- standalone scores: each worker against the empty placement
  res.standalone.assign(m, 0);
  std::vector<ChainState> hs(slots);
  for (int32_t lo = 0; lo < m; lo += kMaxChains) {
    const int32_t hi = std::min(m, lo + kMaxChains);
    std::vector<int32_t> sl, wk, kk;
    for (int32_t h = lo; h < hi; ++h) {
      sl.push_back(h);
      wk.push_back(h);
      kk.push_back(kp[h]);
    }
    ChainSet all = chain_set(sl, wk, kk, 0, sl.size());
    PP_HIP(launch_init_slots(all, d, 1, st));
    PP_HIP(launch_gains(all, d, st));
    std::vector<int32_t> sl2, wk2, kk2;
    for (size_t q = 0; q < sl.size(); ++q)
      if (kk[q] > 0) {
        sl2.push_back(sl[q]);
        wk2.push_back(wk[q]);
        kk2.push_back(kk[q]);
      }
    if (!sl2.empty()) {
      // the choice bits and the walk too: every start's first greedy update
      // is the standalone solve of its first worker
      const ChainSet s2 = chain_set(sl2, wk2, kk2, 0, sl2.size());
      PP_TRY(e.dp(s2, 1));
      PP_HIP(launch_backtrack(s2, d, kModeGreedy, st));
    }
  }
  // the standalone selections (slots 0..m-1) outlive the starts' use of
  // those slots
  const size_t sel_bytes = (size_t)m * (d.npad / 32) * sizeof(uint32_t);
  PP_TRY(c->sel0.ensure(sel_bytes));
  PP_HIP(hipMemcpyAsync(c->sel0.p, d.sel, sel_bytes, hipMemcpyDeviceToDevice, st));
  PP_HIP(hipMemcpyAsync(hs.data(), d.cs, sizeof(ChainState) * m,
                        hipMemcpyDeviceToHost, st));
  PP_TRY(poll_stream(st));
  for (int32_t h = 0; h < m; ++h) {
    if (hs[h].status) return stall_fail();
    res.standalone[h] = kp[h] > 0 ? hs[h].dpval : 0;
  }

  // --- start orders
  res.orders.assign((size_t)S * m, 0);
  if (o.orders)
    std::memcpy(res.orders.data(), o.orders, sizeof(int32_t) * S * m);
  else
    make_orders(m, o.n_starts, o.order_seed, res.standalone.data(),
                res.orders.data());

  // --- starts: WorkerGreedy then refinement sweeps, all starts together
  res.sweeps.assign(S, 0);
  res.accepts.assign(S, 0);
  res.start_obj.assign(S, 0);
  for (int32_t lo = 0; lo < S; lo += kMaxChains) {
    const int32_t hi = std::min(S, lo + kMaxChains);
    std::vector<int32_t> active;
    for (int32_t s = lo; s < hi; ++s) active.push_back(s);
    {
      std::vector<int32_t> sl(active);
      for (int32_t q = spare_base; q < slots; ++q) sl.push_back(q);
      std::vector<int32_t> wk(sl.size(), 0), kk(sl.size(), 0);
      PP_HIP(launch_init_slots(chain_set(sl, wk, kk, 0, sl.size()), d, 1, st));
    }
    auto position_set = [&](const std::vector<int32_t>& act, int32_t a) {
      std::vector<int32_t> sl, wk, kk;
      for (int32_t s : act) {
        const int32_t h = res.orders[(size_t)s * m + a];
        if (kp[h] == 0) continue;  // empty set: never changes the placement
        sl.push_back(s);
        wk.push_back(h);
        kk.push_back(kp[h]);
      }
      return chain_set(sl, wk, kk, 0, sl.size());
    };
    {
      const ChainSet first = position_set(active, 0);
      PP_TRY(e.take_standalone(first, c->sel0.as<uint32_t>()));
      for (int32_t q = 0; q < first.count; ++q) res.skipped_cells += (int64_t)n * first.kprime[q];
    }
    for (int32_t a = 1; a < m; ++a)
      PP_TRY(e.update(position_set(active, a), kModeGreedy));
    if (!(o.flags & PP_F_NO_REFINE))
      PP_TRY(refine_starts(e, active, spare_base, spec_chains,
                           std::min(spec_blocks, e.resident), m, kp,
                           o.max_rounds, res));
    std::vector<int32_t> sl, wk, kk;
    for (int32_t s = lo; s < hi; ++s) {
      sl.push_back(s);
      wk.push_back(0);
      kk.push_back(0);
    }
    ChainSet all = chain_set(sl, wk, kk, 0, sl.size());
    PP_HIP(launch_objective(all, d, st));
    std::vector<ChainState> fin(hi - lo);
    PP_HIP(hipMemcpyAsync(fin.data(), d.cs + lo, sizeof(ChainState) * (hi - lo),
                          hipMemcpyDeviceToHost, st));
    PP_TRY(poll_stream(st));
    for (int32_t s = lo; s < hi; ++s) {
      if (fin[s - lo].status) return stall_fail();
      res.start_obj[s] = fin[s - lo].obj;
      res.accepts[s] = fin[s - lo].accepts;
      res.skipped_cells += fin[s - lo].skipped_cells;
    }
  }
  res.best = 0;
  if (f64) {
    // real-valued costs: starts compare exact objective values
    PP_TRY(read_exact(d, 0, S, st, res.start_gx));
    for (int32_t s = 1; s < S; ++s)
      if (ex_cmp(&res.start_gx[(size_t)s * kExLimbs],
                 &res.start_gx[(size_t)res.best * kExLimbs]) > 0)
        res.best = s;
    res.win_gx.assign(res.start_gx.begin() + (size_t)res.best * kExLimbs,
                      res.start_gx.begin() + (size_t)(res.best + 1) * kExLimbs);
  } else {
    for (int32_t s = 1; s < S; ++s)
      if (res.start_obj[s] > res.start_obj[res.best]) res.best = s;
  }
  res.win_slot = res.best;
  res.win_obj = res.start_obj[res.best];
  res.updates = m;
  res.cells = cells_pass;
  for (int32_t s = 0; s < S; ++s) {
    res.updates += (int64_t)m * (1 + res.sweeps[s]);
    res.cells += cells_pass * (1 + res.sweeps[s]);
  }
  if (sg_asked) PP_TRY(run_safeguards(e, m, kp, slot_b, cells_pass, st, res));
  if (e.timer.on) {
    float tot = 0.f;
    for (auto& mk : e.timer.marks) {
      float ms = 0.f;
      PP_HIP(hipEventElapsedTime(&ms, mk.first, mk.second));
      tot += ms;
    }
    res.dp_ms = tot;
    res.dp_launches = (int32_t)e.timer.marks.size();
  }
  return PP_OK;
}

// ---------------------------------------------------------- validation --

int check_options(int32_t m, const pp_options& o) {
  if (o.n_starts < 0 || o.max_rounds < 0)
    return fail(PP_E_ARG, "n_starts and max_rounds must be >= 0");
  if (o.orders) {
    if (o.n_starts < 1)
      return fail(PP_E_ARG, "explicit orders need n_starts >= 1");
    for (int32_t s = 0; s < o.n_starts; ++s) {
      std::vector<char> seen(m, 0);
      for (int32_t a = 0; a < m; ++a) {
        const int32_t h = o.orders[(size_t)s * m + a];
        if (h < 0 || h >= m || seen[h])
          return fail(PP_E_ARG, "orders[" + std::to_string(s) +
                                    "] is not a permutation of 0..m-1");
        seen[h] = 1;
      }
    }
  }
  return PP_OK;
}

int check_values(int32_t n, int32_t m, const int64_t* lam, const int64_t* w,
                 const int64_t* f, unsigned __int128* total = nullptr) {
  const size_t mn = (size_t)m * n;
  for (size_t x = 0; x < mn; ++x)
    if (lam[x] < 0 || w[x] < 0)
      return fail(PP_E_RANGE, "negative demand or recompute cost");
  for (size_t x = 0; x < mn * (size_t)m; ++x)
    if (f[x] < 0) return fail(PP_E_RANGE, "negative fetch cost");
  unsigned __int128 tot = 0;
  for (size_t x = 0; x < mn; ++x) {
    tot += (unsigned __int128)(uint64_t)lam[x] * (uint64_t)w[x];
    if (tot > (unsigned __int128)INT64_MAX)
      return fail(PP_E_OVERFLOW, "sum of demand * recompute cost exceeds INT64_MAX");
  }
  if (total) *total = tot;
  return PP_OK;
}

// Real-valued inputs: finite and non-negative (NaN fails every comparison).
bool finite_nonneg(double x) { return x >= 0.0 && x <= DBL_MAX; }

int check_values_f64(int32_t n, int32_t m, const double* lam, const double* w,
                     const double* f) {
  const size_t mn = (size_t)m * n;
  for (size_t x = 0; x < mn; ++x)
    if (!finite_nonneg(lam[x]) || !finite_nonneg(w[x]))
      return fail(PP_E_RANGE, "demand and recompute cost must be finite and >= 0");
  for (size_t x = 0; x < mn * (size_t)m; ++x)
    if (!finite_nonneg(f[x]))
      return fail(PP_E_RANGE, "fetch cost must be finite and >= 0");
  return PP_OK;
}

int check_f64_options(double eps) {
  if (!finite_nonneg(eps)) return fail(PP_E_ARG, "epsilon must be finite and >= 0");
  return PP_OK;
}

// Every marginal, DP value and objective is at most sum Lambda*w; below
// 2^62 the sweep may take its maximum with v_max_f64 on the bit patterns.
constexpr unsigned __int128 kFmaxBound = (unsigned __int128)1 << 62;

int check_common(int32_t n, int32_t m, const void* a, const void* b,
                 const void* c2, const void* d2) {
  if (n < 1) return fail(PP_E_ARG, "n must be >= 1");
  if (m < 1 || m > 255) return fail(PP_E_ARG, "m must be in 1..255");
  if (!a || !b || !c2 || !d2) return fail(PP_E_ARG, "null pointer argument");
  return PP_OK;
}

pp_options default_options() {
  pp_options o;
  o.n_starts = 8;
  o.max_rounds = 0;
  o.order_seed = 0;
  o.orders = nullptr;
  o.flags = 0;
  return o;
}

// Per-thread default context for the host-pointer entry points.
pp_ctx* thread_ctx(int& rc) {
  thread_local std::unique_ptr<pp_ctx> ctx;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    rc = fail(PP_E_DEVICE, "no HIP device");
    return nullptr;
  }
  if (!ctx || ctx->device != dev) {
    ctx.reset();
    pp_ctx* c = nullptr;
    rc = pp_ctx_create(&c, dev);
    if (rc != PP_OK) return nullptr;
    ctx.reset(c);
  }
  rc = PP_OK;
  return ctx.get();
}

// Upload the tree layout and (already gathered or identity) inputs.
int upload_tree(pp_ctx* c, const TreeLayout& t, hipStream_t st) {
  const size_t n = (size_t)t.n;
  const size_t a = (n * 4 + 255) & ~(size_t)255, ceb = t.ce.size() * 4;
  std::vector<uint8_t>& h = c->tree_host;
  h.assign(2 * a + ceb, 0);
  std::memcpy(h.data(), t.nextpos.data(), n * 4);
  std::memcpy(h.data() + a, t.order.data(), n * 4);
  std::memcpy(h.data() + 2 * a, t.ce.data(), ceb);
  PP_TRY(c->tree.ensure(h.size()));
  c->nextpos = c->tree.as<int32_t>();
  c->order = (int32_t*)(c->tree.as<uint8_t>() + a);
  c->ce = (uint32_t*)(c->tree.as<uint8_t>() + 2 * a);
  return stage_h2d(c, c->tree.p, h.data(), h.size(), st);
}

// Every LDS row the metadata names must lie inside the sweep's LDS layout.
int check_meta(const TreeLayout& t, const std::vector<uint32_t>& meta,
               int cells) {
  if (t.leaf.empty() || !t.leaf[0])
    return fail(PP_E_DEVICE, "internal: the first DP step must be a leaf");
  const int64_t row = dp_row_stride(cells);
  if (meta.size() != kMetaWords * t.leaf.size() || meta[2] != 0xFFFFFFFFu)
    return fail(PP_E_DEVICE, "internal: DP step metadata malformed");
  const int64_t h = t.slots;
  for (size_t q = 0; q < meta.size(); q += kMetaWords) {
    const int64_t st = meta[q], pf = meta[q + 1];
    // stores go to a slot or a sink row, never to the zero row; reads come
    // from a slot or the zero row; the sweep packs both offsets, divided by
    // 8, into the two 16-bit halves of one word
    const bool st_ok = st % row == 0 && (st / row < h ||
                                         (st / row > h && st / row <= h + dp_sink_rows(cells)));
    if (!st_ok || pf % row != 0 || pf / row > h || st >= (8 << 16) || pf >= (8 << 16) ||
        (meta[q + 2] != 0u && meta[q + 2] != 0xFFFFFFFFu) || meta[q + 3] != 0u)
      return fail(PP_E_DEVICE, "internal: DP step metadata out of range");
  }
  return PP_OK;
}

// Deep trees: the sweep's spill lists and the spilled rows' device memory
// for `slots` chain slots of d.stages stages at d.cells cells per lane.
int upload_spills(pp_ctx* c, const TreeLayout& t, DevState& d, int32_t slots,
                  hipStream_t st) {
  d.nspill = t.nspill;
  d.sp_out_off = d.sp_out = d.sp_in_off = d.sp_in = nullptr;
  d.spill = nullptr;
  if (t.nspill == 0) return PP_OK;
  const size_t a = t.out_off.size(), b = t.spill_out.size(), c2 = t.in_off.size(),
               e = t.spill_in.size();
  PP_TRY(c->sp_lists.ensure((a + b + c2 + e) * 4));
  int32_t* base = c->sp_lists.as<int32_t>();
  PP_TRY(stage_h2d(c, base, t.out_off.data(), a * 4, st));
  PP_TRY(stage_h2d(c, base + a, t.spill_out.data(), b * 4, st));
  PP_TRY(stage_h2d(c, base + a + b, t.in_off.data(), c2 * 4, st));
  PP_TRY(stage_h2d(c, base + a + b + c2, t.spill_in.data(), e * 4, st));
  d.sp_out_off = base;
  d.sp_out = base + a;
  d.sp_in_off = base + a + b;
  d.sp_in = base + a + b + c2;
  PP_TRY(c->spill.ensure((size_t)slots * d.stages * t.nspill * 64 * d.cells * 8));
  d.spill = c->spill.as<uint64_t>();
  return PP_OK;
}

int upload_meta(pp_ctx* c, const TreeLayout& t, int cells, hipStream_t st) {
  c->meta_host = encode_meta(t, cells);
  PP_TRY(check_meta(t, c->meta_host, cells));
  PP_TRY(c->meta.ensure(c->meta_host.size() * 4));
  PP_TRY(stage_h2d(c, c->meta.p, c->meta_host.data(), c->meta_host.size() * 4, st));
  return PP_OK;
}

// Device inputs in caller ids -> context buffers in preorder.
int layout_inputs(pp_ctx* c, const TreeLayout& t, int32_t m,
                  const int64_t* lam, const int64_t* w, const int64_t* f,
                  hipStream_t st) {
  const size_t n = (size_t)t.n;
  PP_TRY(c->lam.ensure(m * n * 8));
  PP_TRY(c->w.ensure(m * n * 8));
  PP_TRY(c->f.ensure((size_t)m * m * n * 8));
  const int32_t* ord = c->order;
  PP_HIP(launch_gather_inputs(lam, w, f, c->lam.as<int64_t>(), c->w.as<int64_t>(),
                              c->f.as<int64_t>(), m, t.n, ord, st));
  return PP_OK;
}

void fill_stats(pp_stats* stats, const PlanResult& r, int32_t m) {
  if (!stats) return;
  stats->best_start = r.best;
  stats->n_starts = r.S;
  stats->updates = r.updates;
  stats->dp_cells = r.cells;
  if (stats->start_objective)
    std::copy(r.start_obj.begin(), r.start_obj.end(), stats->start_objective);
  if (stats->start_sweeps)
    std::copy(r.sweeps.begin(), r.sweeps.end(), stats->start_sweeps);
  if (stats->start_accepts)
    std::copy(r.accepts.begin(), r.accepts.end(), stats->start_accepts);
  if (stats->standalone)
    std::copy(r.standalone.begin(), r.standalone.end(), stats->standalone);
  if (stats->orders) std::copy(r.orders.begin(), r.orders.end(), stats->orders);
  stats->dp_kernel_ms = r.dp_ms;
  stats->dp_launches = r.dp_launches;
  stats->safeguards_run = r.sg_run ? 1 : 0;
  for (int q = 0; q < 3; ++q) stats->safeguard_objective[q] = r.sg_obj[q];
  stats->dp_cells_executed = r.cells - r.skipped_cells + r.spec_cells;
  stats->dp_lane_cells = r.lane_cells;
  stats->dp_fmax = r.fmax;
  stats->dp_restarts = r.restarts;
  (void)m;
}

double bits_f64(int64_t v) {
  double d;
  std::memcpy(&d, &v, sizeof d);
  return d;
}

void fill_stats_f64(pp_stats_f64* stats, const PlanResult& r) {
  if (!stats) return;
  stats->best_start = r.best;
  stats->n_starts = r.S;
  stats->updates = r.updates;
  stats->dp_cells = r.cells;
  if (stats->start_objective)
    for (size_t s = 0; s < r.start_obj.size(); ++s)
      stats->start_objective[s] = bits_f64(r.start_obj[s]);
  if (stats->start_sweeps)
    std::copy(r.sweeps.begin(), r.sweeps.end(), stats->start_sweeps);
  if (stats->start_accepts)
    std::copy(r.accepts.begin(), r.accepts.end(), stats->start_accepts);
  if (stats->standalone)
    for (size_t h = 0; h < r.standalone.size(); ++h)
      stats->standalone[h] = bits_f64(r.standalone[h]);
  if (stats->orders) std::copy(r.orders.begin(), r.orders.end(), stats->orders);
  stats->dp_kernel_ms = r.dp_ms;
  stats->dp_launches = r.dp_launches;
  stats->safeguards_run = r.sg_run ? 1 : 0;
  for (int q = 0; q < 3; ++q) stats->safeguard_objective[q] = bits_f64(r.sg_obj[q]);
  stats->dp_cells_executed = r.cells - r.skipped_cells + r.spec_cells;
  stats->dp_lane_cells = r.lane_cells;
  stats->dp_fmax = r.fmax;
  stats->dp_restarts = r.restarts;
}

// Host-array inputs (caller ids, 8-byte values) to the context's preorder
// layout: upload, tree tables, gather.
int upload_host_inputs(pp_ctx* c, const TreeLayout& t, int32_t m, const void* demand,
                       const void* recompute_cost, const void* fetch_cost,
                       hipStream_t st) {
  const size_t mn = (size_t)m * t.n;
  PP_TRY(c->up_lam.ensure(mn * 8));
  PP_TRY(c->up_w.ensure(mn * 8));
  PP_TRY(c->up_f.ensure(mn * m * 8));
  PP_HIP(hipMemcpyAsync(c->up_lam.p, demand, mn * 8, hipMemcpyHostToDevice, st));
  PP_HIP(hipMemcpyAsync(c->up_w.p, recompute_cost, mn * 8, hipMemcpyHostToDevice, st));
  PP_HIP(hipMemcpyAsync(c->up_f.p, fetch_cost, mn * m * 8, hipMemcpyHostToDevice, st));
  PP_TRY(upload_tree(c, t, st));
  return layout_inputs(c, t, m, c->up_lam.as<int64_t>(), c->up_w.as<int64_t>(),
                       c->up_f.as<int64_t>(), st);
}

// Slot `slot`'s placement (preorder) to host memory in caller ids.
int placement_to_host(pp_ctx* c, const TreeLayout& t, int32_t m, int32_t slot,
                      uint8_t* out, hipStream_t st) {
  const size_t n = (size_t)t.n, mn = (size_t)m * n;
  std::vector<uint8_t> pre(mn);
  PP_HIP(hipMemcpyAsync(pre.data(), c->tgt.as<uint8_t>() + (size_t)slot * mn, mn,
                        hipMemcpyDeviceToHost, st));
  PP_TRY(poll_stream(st));
  for (int32_t h = 0; h < m; ++h)
    for (size_t q = 0; q < n; ++q) out[(size_t)h * n + t.order[q]] = pre[(size_t)h * n + q];
  return PP_OK;
}

// Re-planning, after run_plan with one spare slot: the incumbent (caller
// ids) into that slot, its objective under the refreshed inputs (Eq. 6) and
// the one-time cost of the proposal's new (worker, chunk) pairs, summed
// exactly (integers) or in a fixed order (doubles).
struct ReplanEval {
  int64_t g_inc = 0;              // objective bits
  unsigned __int128 cost = 0;     // integer costs
  // real-valued costs: the exact cost and the exact G(T') - G(T), each
  // rounded to the nearest double
  double cost_f64 = 0.0;
  double gain_f64 = 0.0;
};

int replan_evaluate(pp_ctx* c, const TreeLayout& t, int32_t m, const PlanResult& r,
                    const uint8_t* incumbent, bool f64, double eps, hipStream_t st,
                    ReplanEval& ev) {
  const int32_t n = t.n;
  const size_t mn = (size_t)m * n;
  DevState d{};
  d.n = n;
  d.m = m;
  d.npad = npad_of(n);
  d.lam = c->lam.as<int64_t>();
  d.w = c->w.as<int64_t>();
  d.f = c->f.as<int64_t>();
  d.tgt = c->tgt.as<uint8_t>();
  d.v1 = c->v1.as<int64_t>();
  d.v2 = c->v2.as<int64_t>();
  d.h1 = c->h1.as<uint8_t>();
  d.cs = c->cs.as<ChainState>();
  if (f64) {
    d.f64 = 1;
    d.eps = eps;
    d.gx_blocks = gexact_blocks(n, m);
    d.gx = c->gx.as<uint32_t>();
    d.gxp = c->gxp.as<uint64_t>();
  }
  const int32_t xs = r.extra_slot;
  std::vector<uint8_t> pre(mn);
  for (int32_t h = 0; h < m; ++h)
    for (int32_t q = 0; q < n; ++q)
      pre[(size_t)h * n + q] = incumbent[(size_t)h * n + t.order[q]];
  PP_HIP(hipMemcpyAsync(d.tgt + (size_t)xs * mn, pre.data(), mn,
                        hipMemcpyHostToDevice, st));
  const std::vector<int32_t> one = {xs}, zero = {0};
  const ChainSet inc_set = chain_set(one, zero, zero, 0, 1);
  PP_HIP(launch_init_slots(inc_set, d, 0, st));
  PP_HIP(launch_holder_build(inc_set, d, st));
  PP_HIP(launch_objective(inc_set, d, st));
  const size_t part_bytes = f64 ? (size_t)kExLimbs * 8 : 16;
  PP_TRY(c->partial.ensure(1024 * part_bytes));
  int32_t nb = 0;
  PP_HIP(launch_mat_cost(d, xs, r.win_slot, c->partial.p, &nb, st));
  std::vector<unsigned char> part((size_t)nb * part_bytes);
  ChainState inc_cs{};
  PP_HIP(hipMemcpyAsync(part.data(), c->partial.p, part.size(), hipMemcpyDeviceToHost, st));
  PP_HIP(hipMemcpyAsync(&inc_cs, d.cs + xs, sizeof(ChainState), hipMemcpyDeviceToHost, st));
  PP_TRY(poll_stream(st));
  ev.g_inc = inc_cs.obj;
  if (!f64) {
    for (int32_t b = 0; b < nb; ++b) {
      unsigned __int128 v;
      std::memcpy(&v, part.data() + 16 * (size_t)b, 16);
      ev.cost += v;
    }
    return PP_OK;
  }
  // the exact cost: the blocks' lazy limbs, summed and carried
  std::vector<uint32_t> cost(kExLimbs);
  unsigned __int128 carry = 0;
  for (int q = 0; q < kExLimbs; ++q) {
    unsigned __int128 v = carry;
    for (int32_t b = 0; b < nb; ++b) {
      uint64_t x;
      std::memcpy(&x, part.data() + ((size_t)b * kExLimbs + q) * 8, 8);
      v += x;
    }
    cost[q] = (uint32_t)v;
    carry = v >> 32;
  }
  ev.cost_f64 = bits_f64((int64_t)ex_round_bits(cost.data()));
  // G(T') - G(T), exact, then rounded
  std::vector<uint32_t> ginc, diff(kExLimbs);
  PP_TRY(read_exact(d, xs, 1, st, ginc));
  const uint32_t* gw = r.win_gx.data();
  if (ex_cmp(gw, ginc.data()) >= 0) {
    ex_sub(diff.data(), gw, ginc.data());
    ev.gain_f64 = bits_f64((int64_t)ex_round_bits(diff.data()));
  } else {
    ex_sub(diff.data(), ginc.data(), gw);
    ev.gain_f64 = -bits_f64((int64_t)ex_round_bits(diff.data()));
  }
  return PP_OK;
}

// target := proposal if adopted, else the incumbent; proposal optional.
int replan_outputs(pp_ctx* c, const TreeLayout& t, int32_t m, const PlanResult& r,
                   const uint8_t* incumbent, bool adopt, uint8_t* target,
                   uint8_t* proposal, hipStream_t st) {
  const size_t mn = (size_t)m * t.n;
  std::vector<uint8_t> prop(mn);
  PP_TRY(placement_to_host(c, t, m, r.win_slot, prop.data(), st));
  if (proposal) std::memcpy(proposal, prop.data(), mn);
  std::memcpy(target, adopt ? prop.data() : incumbent, mn);
  return PP_OK;
}

template <class F>
int guarded(F&& fn) {
  try {
    return fn();
  } catch (const std::bad_alloc&) {
    return fail(PP_E_NOMEM, "host allocation failed");
  } catch (...) {
    return fail(PP_E_DEVICE, "unexpected internal exception");
  }
}

}  // namespace

// ================================================================ C ABI ===

extern "C" {

int pp_abi_version(void) { return PP_ABI_VERSION; }

const char* pp_last_error(void) { return g_err; }

int32_t pp_num_starts(int32_t m, int32_t n_starts) {
  return num_starts(m, n_starts);
}

int pp_orders(int32_t m, int32_t n_starts, uint64_t order_seed,
              const int64_t* standalone, int32_t* orders) {
  g_err[0] = 0;
  if (m < 1 || m > 255 || n_starts < 0 || !standalone || !orders)
    return fail(PP_E_ARG, "bad arguments to pp_orders");
  return guarded([&] {
    make_orders(m, n_starts, order_seed, standalone, orders);
    return PP_OK;
  });
}

int pp_sweep_layout(int32_t n, const int32_t* parent, int32_t cells,
                    uint32_t* meta, int32_t* nsteps, int32_t* slots) {
  g_err[0] = 0;
  return guarded([&]() -> int {
    if (n < 1 || !parent || !nsteps || !slots)
      return fail(PP_E_ARG, "bad arguments to pp_sweep_layout");
    if (cells != 1 && cells != 2 && cells != 4)
      return fail(PP_E_ARG, "cells must be 1, 2 or 4");
    TreeLayout t;
    PP_TRY(build_tree(n, parent, t));
    const std::vector<uint32_t> mv = encode_meta(t, cells);
    PP_TRY(check_meta(t, mv, cells));
    if (meta) std::copy(mv.begin(), mv.end(), meta);
    *nsteps = (int32_t)(mv.size() / kMetaWords);
    *slots = t.slots;
    return PP_OK;
  });
}

static_assert(kCeEnd == PP_BT_END, "one end marker for the backtrack table");
static_assert(kNoAllocScratchBytes == PP_NOALLOC_SCRATCH_BYTES, "one scratch size");

int pp_sweep_spills(int32_t n, const int32_t* parent, int32_t* nbatches, int32_t* nspill,
                    int32_t* n_out, int32_t* n_in, int32_t* out_off, int32_t* spill_out,
                    int32_t* in_off, int32_t* spill_in) {
  g_err[0] = 0;
  return guarded([&]() -> int {
    if (n < 1 || !parent || !nbatches || !nspill || !n_out || !n_in)
      return fail(PP_E_ARG, "null pointer or n < 1");
    TreeLayout t;
    PP_TRY(build_tree(n, parent, t));
    const int32_t nb = (int32_t)(t.leaf.size() / kDpBatch);
    *nbatches = nb;
    *nspill = t.nspill;
    *n_out = (int32_t)t.spill_out.size() / 2;
    *n_in = (int32_t)t.spill_in.size() / 2;
    if (t.nspill == 0) {
      if (out_off) std::fill(out_off, out_off + nb + 1, 0);
      if (in_off) std::fill(in_off, in_off + nb + 1, 0);
      return PP_OK;
    }
    if (out_off) std::copy(t.out_off.begin(), t.out_off.end(), out_off);
    if (in_off) std::copy(t.in_off.begin(), t.in_off.end(), in_off);
    if (spill_out) std::copy(t.spill_out.begin(), t.spill_out.end(), spill_out);
    if (spill_in) std::copy(t.spill_in.begin(), t.spill_in.end(), spill_in);
    return PP_OK;
  });
}

int pp_backtrack_table(int32_t n, const int32_t* parent, uint32_t* table,
                       int64_t* rows) {
  g_err[0] = 0;
  return guarded([&]() -> int {
    if (n < 1 || !parent || !rows) return fail(PP_E_ARG, "bad arguments to pp_backtrack_table");
    TreeLayout t;
    PP_TRY(build_tree(n, parent, t));
    if (table) std::copy(t.ce.begin(), t.ce.end(), table);
    *rows = (int64_t)(t.ce.size() / 4);
    return PP_OK;
  });
}

int pp_ctx_create(pp_ctx** ctx, int device) {
  g_err[0] = 0;
  if (!ctx) return fail(PP_E_ARG, "null ctx");
  return guarded([&]() -> int {
    int count = 0;
    if (hipGetDeviceCount(&count) != hipSuccess || count < 1)
      return fail(PP_E_DEVICE, "no HIP device");
    if (device < 0 || device >= count) return fail(PP_E_ARG, "bad device index");
    std::unique_ptr<pp_ctx> c(new pp_ctx);
    c->device = device;
    PP_TRY(select_device(c.get()));
    PP_HIP(hipStreamCreateWithFlags(&c->own, hipStreamNonBlocking));
    *ctx = c.release();
    return PP_OK;
  });
}

void pp_ctx_destroy(pp_ctx* ctx) {
  if (!ctx) return;
  (void)hipSetDevice(ctx->device);
  (void)hipDeviceSynchronize();
  delete ctx;
}

int pp_plan_device(pp_ctx* ctx, int32_t n, int32_t m, const int32_t* parent,
                   const int64_t* demand_dev, const int64_t* recompute_dev,
                   const int64_t* fetch_dev, const int32_t* cap,
                   const pp_options* opt, uint8_t* target_dev,
                   int64_t* objective, pp_stats* stats, void* hip_stream) {
  g_err[0] = 0;
  return guarded([&]() -> int {
    if (!ctx) return fail(PP_E_ARG, "null ctx");
    PP_TRY(check_common(n, m, parent, demand_dev, recompute_dev, fetch_dev));
    if (!cap || !target_dev || !objective) return fail(PP_E_ARG, "null pointer argument");
    const pp_options o = opt ? *opt : default_options();
    PP_TRY(check_options(m, o));
    for (int32_t h = 0; h < m; ++h)
      if (cap[h] < 0) return fail(PP_E_RANGE, "negative capacity");
    TreeLayout t;
    if (o.flags & PP_F_VALIDATE_ONLY) return build_tree(n, parent, t);
    PP_TRY(select_device(ctx));
    hipStream_t st = (hipStream_t)hip_stream;
    // value checks on the device (negatives, and the sum of lam*w added
    // exactly), while the host builds the tree tables
    PP_TRY(ctx->partial.ensure(2 * kValidateBlocks * 8));
    PP_TRY(ensure_val_pin(ctx));
    int32_t nb = 0;
    PP_HIP(launch_validate(demand_dev, recompute_dev, fetch_dev, n, m,
                           ctx->partial.as<uint64_t>(), &nb, st));
    PP_HIP(hipMemcpyAsync(ctx->val_pin, ctx->partial.p, 16 * (size_t)nb,
                          hipMemcpyDeviceToHost, st));
    const int trc = build_tree(n, parent, t);
    if (trc != PP_OK) {
      PP_TRY(poll_stream(st));
      return trc;
    }
    // the layout does not depend on the checks' outcome
    PP_TRY(upload_tree(ctx, t, st));
    PP_TRY(layout_inputs(ctx, t, m, demand_dev, recompute_dev, fetch_dev, st));
    PP_TRY(poll_stream(st));
    unsigned __int128 tot = 0;
    for (int32_t b = 0; b < nb; ++b) {
      if (ctx->val_pin[nb + b]) return fail(PP_E_RANGE, "negative demand or cost");
      tot += ctx->val_pin[b];
    }
    if (tot > (unsigned __int128)INT64_MAX)
      return fail(PP_E_OVERFLOW, "sum of demand * recompute cost exceeds INT64_MAX");
    PlanResult r;
    PP_TRY(run_plan(ctx, t, m, cap, o, tot < kFmaxBound, st, r));
    // best start's placement back to caller ids
    const size_t mn = (size_t)m * n;
    PP_HIP(launch_scatter_u8(ctx->tgt.as<uint8_t>() + (size_t)r.win_slot * mn,
                             target_dev, m, n, ctx->order, st));
    PP_TRY(poll_stream(st));
    *objective = r.win_obj;
    fill_stats(stats, r, m);
    return PP_OK;
  });
}

int pp_plan(int32_t n, int32_t m, const int32_t* parent, const int64_t* demand,
            const int64_t* recompute_cost, const int64_t* fetch_cost,
            const int32_t* cap, const pp_options* opt, uint8_t* target,
            int64_t* objective, pp_stats* stats) {
  g_err[0] = 0;
  return guarded([&]() -> int {
    PP_TRY(check_common(n, m, parent, demand, recompute_cost, fetch_cost));
    if (!cap || !target || !objective) return fail(PP_E_ARG, "null pointer argument");
    const pp_options o = opt ? *opt : default_options();
    PP_TRY(check_options(m, o));
    for (int32_t h = 0; h < m; ++h)
      if (cap[h] < 0) return fail(PP_E_RANGE, "negative capacity");
    unsigned __int128 tot = 0;
    PP_TRY(check_values(n, m, demand, recompute_cost, fetch_cost, &tot));
    TreeLayout t;
    PP_TRY(build_tree(n, parent, t));
    if (o.flags & PP_F_VALIDATE_ONLY) return PP_OK;
    int rc = PP_OK;
    pp_ctx* c = thread_ctx(rc);
    if (!c) return rc;
    hipStream_t st = c->own;
    PP_TRY(upload_host_inputs(c, t, m, demand, recompute_cost, fetch_cost, st));
    PlanResult r;
    PP_TRY(run_plan(c, t, m, cap, o, tot < kFmaxBound, st, r));
    PP_TRY(placement_to_host(c, t, m, r.win_slot, target, st));
    *objective = r.win_obj;
    fill_stats(stats, r, m);
    return PP_OK;
  });
}

int pp_plan_f64_device(pp_ctx* ctx, int32_t n, int32_t m, const int32_t* parent,
                       const double* demand_dev, const double* recompute_dev,
                       const double* fetch_dev, const int32_t* cap, double epsilon,
                       const pp_options* opt, uint8_t* target_dev, double* objective,
                       pp_stats_f64* stats, void* hip_stream) {
  g_err[0] = 0;
  return guarded([&]() -> int {
    if (!ctx) return fail(PP_E_ARG, "null ctx");
    PP_TRY(check_common(n, m, parent, demand_dev, recompute_dev, fetch_dev));
    if (!cap || !target_dev || !objective) return fail(PP_E_ARG, "null pointer argument");
    const pp_options o = opt ? *opt : default_options();
    PP_TRY(check_options(m, o));
    PP_TRY(check_f64_options(epsilon));
    for (int32_t h = 0; h < m; ++h)
      if (cap[h] < 0) return fail(PP_E_RANGE, "negative capacity");
    TreeLayout t;
    if (o.flags & PP_F_VALIDATE_ONLY) return build_tree(n, parent, t);
    PP_TRY(select_device(ctx));
    hipStream_t st = (hipStream_t)hip_stream;
    // value checks on the device while the host builds the tree tables
    PP_TRY(ctx->partial.ensure(2 * kValidateBlocks * 8));
    PP_TRY(ensure_val_pin(ctx));
    int32_t nb = 0;
    PP_HIP(launch_validate_f64(demand_dev, recompute_dev, fetch_dev, n, m,
                               ctx->partial.as<uint64_t>(), &nb, st));
    PP_HIP(hipMemcpyAsync(ctx->val_pin, ctx->partial.p, 8 * (size_t)nb,
                          hipMemcpyDeviceToHost, st));
    const int trc = build_tree(n, parent, t);
    if (trc != PP_OK) {
      PP_TRY(poll_stream(st));
      return trc;
    }
    // the layout does not depend on the checks' outcome
    PP_TRY(upload_tree(ctx, t, st));
    PP_TRY(layout_inputs(ctx, t, m, (const int64_t*)demand_dev,
                         (const int64_t*)recompute_dev, (const int64_t*)fetch_dev, st));
    PP_TRY(poll_stream(st));
    for (int32_t b = 0; b < nb; ++b)
      if (ctx->val_pin[b]) return fail(PP_E_RANGE, "demand and costs must be finite and >= 0");
    PlanResult r;
    PP_TRY(run_plan(ctx, t, m, cap, o, false, st, r, 0, true, epsilon));
    const size_t mn = (size_t)m * n;
    PP_HIP(launch_scatter_u8(ctx->tgt.as<uint8_t>() + (size_t)r.win_slot * mn,
                             target_dev, m, n, ctx->order, st));
    PP_TRY(poll_stream(st));
    *objective = bits_f64(r.win_obj);
    fill_stats_f64(stats, r);
    return PP_OK;
  });
}

int pp_plan_f64(int32_t n, int32_t m, const int32_t* parent, const double* demand,
                const double* recompute_cost, const double* fetch_cost,
                const int32_t* cap, double epsilon, const pp_options* opt,
                uint8_t* target, double* objective, pp_stats_f64* stats) {
  g_err[0] = 0;
  return guarded([&]() -> int {
    PP_TRY(check_common(n, m, parent, demand, recompute_cost, fetch_cost));
    if (!cap || !target || !objective) return fail(PP_E_ARG, "null pointer argument");
    const pp_options o = opt ? *opt : default_options();
    PP_TRY(check_options(m, o));
    PP_TRY(check_f64_options(epsilon));
    for (int32_t h = 0; h < m; ++h)
      if (cap[h] < 0) return fail(PP_E_RANGE, "negative capacity");
    PP_TRY(check_values_f64(n, m, demand, recompute_cost, fetch_cost));
    TreeLayout t;
    PP_TRY(build_tree(n, parent, t));
    if (o.flags & PP_F_VALIDATE_ONLY) return PP_OK;
    int rc = PP_OK;
    pp_ctx* c = thread_ctx(rc);
    if (!c) return rc;
    hipStream_t st = c->own;
    PP_TRY(upload_host_inputs(c, t, m, demand, recompute_cost, fetch_cost, st));
    PlanResult r;
    PP_TRY(run_plan(c, t, m, cap, o, false, st, r, 0, true, epsilon));
    PP_TRY(placement_to_host(c, t, m, r.win_slot, target, st));
    *objective = bits_f64(r.win_obj);
    fill_stats_f64(stats, r);
    return PP_OK;
  });
}

int pp_replan(int32_t n, int32_t m, const int32_t* parent, const int64_t* demand,
              const int64_t* recompute_cost, const int64_t* fetch_cost,
              const int32_t* cap, const uint8_t* incumbent, int64_t horizon,
              const pp_options* opt, uint8_t* target, uint8_t* proposal,
              pp_replan_info* info, pp_stats* stats) {
  g_err[0] = 0;
  return guarded([&]() -> int {
    PP_TRY(check_common(n, m, parent, demand, recompute_cost, fetch_cost));
    if (!cap || !incumbent || !target || !info)
      return fail(PP_E_ARG, "null pointer argument");
    if (horizon < 0) return fail(PP_E_ARG, "horizon must be >= 0");
    const pp_options o = opt ? *opt : default_options();
    PP_TRY(check_options(m, o));
    for (int32_t h = 0; h < m; ++h)
      if (cap[h] < 0) return fail(PP_E_RANGE, "negative capacity");
    const size_t mn = (size_t)m * n;
    for (size_t x = 0; x < mn; ++x)
      if (incumbent[x] > 1) return fail(PP_E_ARG, "incumbent entries must be 0 or 1");
    unsigned __int128 tot = 0;
    PP_TRY(check_values(n, m, demand, recompute_cost, fetch_cost, &tot));
    TreeLayout t;
    PP_TRY(build_tree(n, parent, t));
    if (o.flags & PP_F_VALIDATE_ONLY) return PP_OK;
    int rc = PP_OK;
    pp_ctx* c = thread_ctx(rc);
    if (!c) return rc;
    hipStream_t st = c->own;
    PP_TRY(upload_host_inputs(c, t, m, demand, recompute_cost, fetch_cost, st));
    // the proposal: Algorithm 1 on the refreshed inputs, one slot spare
    PlanResult r;
    PP_TRY(run_plan(c, t, m, cap, o, tot < kFmaxBound, st, r, 1));
    ReplanEval ev;
    PP_TRY(replan_evaluate(c, t, m, r, incumbent, false, 0.0, st, ev));
    const unsigned __int128 cost = ev.cost;
    if (cost > (unsigned __int128)INT64_MAX)
      return fail(PP_E_OVERFLOW, "materialization cost exceeds INT64_MAX");
    // adopt iff horizon * (G(T') - G(T)) > cost, exactly
    const int64_t g_inc = ev.g_inc, g_new = r.win_obj;
    bool adopt = false;
    if (g_new > g_inc)
      adopt = (unsigned __int128)(uint64_t)(g_new - g_inc) * (uint64_t)horizon > cost;
    PP_TRY(replan_outputs(c, t, m, r, incumbent, adopt, target, proposal, st));
    info->adopt = adopt ? 1 : 0;
    info->incumbent_objective = g_inc;
    info->proposal_objective = g_new;
    info->materialization_cost = (int64_t)cost;
    fill_stats(stats, r, m);
    return PP_OK;
  });
}

static int rooted_dp_impl(int32_t n, const int32_t* parent, const void* profit_v,
                          int32_t k, uint8_t* selected, int64_t* value, bool f64) {
  g_err[0] = 0;
  return guarded([&]() -> int {
    if (n < 1) return fail(PP_E_ARG, "n must be >= 1");
    if (!parent || !profit_v || !selected || !value)
      return fail(PP_E_ARG, "null pointer argument");
    if (k < 0) return fail(PP_E_RANGE, "negative capacity");
    const int64_t* profit = (const int64_t*)profit_v;
    unsigned __int128 tot = 0;
    if (f64) {
      for (int32_t b = 0; b < n; ++b)
        if (!finite_nonneg(((const double*)profit_v)[b]))
          return fail(PP_E_RANGE, "profits must be finite and >= 0");
    } else {
      for (int32_t b = 0; b < n; ++b) {
        if (profit[b] < 0) return fail(PP_E_RANGE, "negative profit");
        tot += (uint64_t)profit[b];
      }
      if (tot > (unsigned __int128)INT64_MAX)
        return fail(PP_E_OVERFLOW, "sum of profits exceeds INT64_MAX");
    }
    TreeLayout t;
    PP_TRY(build_tree(n, parent, t));
    const int32_t kp = std::min(k, n);
    if (kp == 0) {
      std::memset(selected, 0, n);
      *value = 0;
      return PP_OK;
    }
    int rc = PP_OK;
    pp_ctx* c = thread_ctx(rc);
    if (!c) return rc;
    hipStream_t st = c->own;
    PP_TRY(upload_tree(c, t, st));
    DevState d{};
    d.n = n;
    d.m = 1;
    d.npad = npad_of(n);
    d.nextpos = c->nextpos;
    d.ce = c->ce;
    d.f64 = f64 ? 1 : 0;
    const int32_t slots_lds = t.slots;
    const int cells = choose_cells((kp + 63) / 64, c->device, slots_lds);
    PP_TRY(ensure_slots(c, d, 1, kp, cells));
    PP_TRY(upload_meta(c, t, cells, st));
    d.meta = c->meta.as<uint32_t>();  // upload_meta may have (re)allocated it
    PP_TRY(upload_spills(c, t, d, 1, st));
    PP_TRY(c->up_lam.ensure((size_t)n * 8));
    PP_HIP(hipMemcpyAsync(c->up_lam.p, profit, (size_t)n * 8, hipMemcpyHostToDevice, st));
    PP_HIP(launch_gather(c->up_lam.as<int64_t>(), d.profit, 1, n,
                         c->order, st));
    std::vector<int32_t> sl{0}, wk{0}, kk{kp};
    ChainSet set = chain_set(sl, wk, kk, 0, 1);
    Engine e;
    e.c = c;
    e.d = d;
    e.st = st;
    e.slots_lds = slots_lds;
    e.resident = dp_resident_blocks(cells, slots_lds, c->device);
    e.fmax = tot < kFmaxBound && env_int("PP_DP_NO_FMAX", 0) == 0;
    if (e.resident <= 0) return fail(PP_E_UNSUPPORTED, "DP sweep cannot be resident");
    std::vector<uint32_t> pre(d.npad / 32);
    ChainState out{};
    for (int attempt = 0;; ++attempt) {  // again, with a longer wait, if it stalled
      e.spin_limit = spin_limit_for(attempt);
      ChainState z{};
      PP_HIP(hipMemcpyAsync(d.cs, &z, sizeof z, hipMemcpyHostToDevice, st));
      PP_TRY(e.dp(set, 1));
      PP_HIP(launch_backtrack(set, d, kModeGreedy, st));
      PP_HIP(hipMemcpyAsync(pre.data(), d.sel, pre.size() * 4, hipMemcpyDeviceToHost, st));
      PP_HIP(hipMemcpyAsync(&out, d.cs, sizeof out, hipMemcpyDeviceToHost, st));
      PP_TRY(poll_stream(st));
      if (!out.status) break;
      if (attempt >= kStallRetries) return stall_fail();
    }
    for (int32_t q = 0; q < n; ++q) selected[t.order[q]] = (pre[q / 32] >> (q % 32)) & 1u;
    *value = out.dpval;
    return PP_OK;
  });
}

int pp_replan_f64(int32_t n, int32_t m, const int32_t* parent, const double* demand,
                  const double* recompute_cost, const double* fetch_cost,
                  const int32_t* cap, const uint8_t* incumbent, double horizon,
                  double epsilon, const pp_options* opt, uint8_t* target,
                  uint8_t* proposal, pp_replan_info_f64* info, pp_stats_f64* stats) {
  g_err[0] = 0;
  return guarded([&]() -> int {
    PP_TRY(check_common(n, m, parent, demand, recompute_cost, fetch_cost));
    if (!cap || !incumbent || !target || !info)
      return fail(PP_E_ARG, "null pointer argument");
    if (!finite_nonneg(horizon)) return fail(PP_E_ARG, "horizon must be finite and >= 0");
    const pp_options o = opt ? *opt : default_options();
    PP_TRY(check_options(m, o));
    PP_TRY(check_f64_options(epsilon));
    for (int32_t h = 0; h < m; ++h)
      if (cap[h] < 0) return fail(PP_E_RANGE, "negative capacity");
    const size_t mn = (size_t)m * n;
    for (size_t x = 0; x < mn; ++x)
      if (incumbent[x] > 1) return fail(PP_E_ARG, "incumbent entries must be 0 or 1");
    PP_TRY(check_values_f64(n, m, demand, recompute_cost, fetch_cost));
    TreeLayout t;
    PP_TRY(build_tree(n, parent, t));
    if (o.flags & PP_F_VALIDATE_ONLY) return PP_OK;
    int rc = PP_OK;
    pp_ctx* c = thread_ctx(rc);
    if (!c) return rc;
    hipStream_t st = c->own;
    PP_TRY(upload_host_inputs(c, t, m, demand, recompute_cost, fetch_cost, st));
    PlanResult r;
    PP_TRY(run_plan(c, t, m, cap, o, false, st, r, 1, true, epsilon));
    ReplanEval ev;
    PP_TRY(replan_evaluate(c, t, m, r, incumbent, true, epsilon, st, ev));
    const double cost = ev.cost_f64;
    const double g_inc = bits_f64(ev.g_inc), g_new = bits_f64(r.win_obj);
    const bool adopt = horizon * ev.gain_f64 > cost;
    PP_TRY(replan_outputs(c, t, m, r, incumbent, adopt, target, proposal, st));
    info->adopt = adopt ? 1 : 0;
    info->incumbent_objective = g_inc;
    info->proposal_objective = g_new;
    info->materialization_cost = cost;
    fill_stats_f64(stats, r);
    return PP_OK;
  });
}

int pp_rooted_dp(int32_t n, const int32_t* parent, const int64_t* profit,
                 int32_t k, uint8_t* selected, int64_t* value) {
  return rooted_dp_impl(n, parent, profit, k, selected, value, false);
}

int pp_rooted_dp_f64(int32_t n, const int32_t* parent, const double* profit,
                     int32_t k, uint8_t* selected, double* value) {
  if (!value) {
    g_err[0] = 0;
    return fail(PP_E_ARG, "null pointer argument");
  }
  int64_t v = 0;
  const int rc = rooted_dp_impl(n, parent, profit, k, selected, &v, true);
  if (rc == PP_OK) *value = bits_f64(v);
  return rc;
}

// pp_marginal / pp_objective: chunks need no tree, so positions = ids.
static int marginal_or_objective(int32_t n, int32_t m, const int64_t* demand,
                                 const int64_t* recompute_cost,
                                 const int64_t* fetch_cost, const uint8_t* target,
                                 int32_t h, int64_t* profit, int64_t* gwo,
                                 int64_t* objective) {
  PP_TRY(check_common(n, m, demand, recompute_cost, fetch_cost, target));
  PP_TRY(check_values(n, m, demand, recompute_cost, fetch_cost));
  int rc = PP_OK;
  pp_ctx* c = thread_ctx(rc);
  if (!c) return rc;
  hipStream_t st = c->own;
  const size_t mn = (size_t)m * n;
  PP_TRY(c->lam.ensure(mn * 8));
  PP_TRY(c->w.ensure(mn * 8));
  PP_TRY(c->f.ensure(mn * m * 8));
  PP_HIP(hipMemcpyAsync(c->lam.p, demand, mn * 8, hipMemcpyHostToDevice, st));
  PP_HIP(hipMemcpyAsync(c->w.p, recompute_cost, mn * 8, hipMemcpyHostToDevice, st));
  PP_HIP(hipMemcpyAsync(c->f.p, fetch_cost, mn * m * 8, hipMemcpyHostToDevice, st));
  DevState d{};
  d.n = n;
  d.m = m;
  d.npad = npad_of(n);
  d.lam = c->lam.as<int64_t>();
  d.w = c->w.as<int64_t>();
  d.f = c->f.as<int64_t>();
  PP_TRY(ensure_slots(c, d, 1, 1, 1));
  std::vector<int32_t> sl{0}, wk{h}, kk{0};
  ChainSet set = chain_set(sl, wk, kk, 0, 1);
  PP_HIP(launch_init_slots(set, d, 0, st));
  PP_HIP(hipMemcpyAsync(d.tgt, target, mn, hipMemcpyHostToDevice, st));
  PP_HIP(launch_holder_build(set, d, st));
  ChainState out{};
  if (profit) {
    PP_HIP(launch_gains(set, d, st));
    PP_HIP(hipMemcpyAsync(profit, d.profit, (size_t)n * 8, hipMemcpyDeviceToHost, st));
  } else {
    PP_HIP(launch_objective(set, d, st));
  }
  PP_HIP(hipMemcpyAsync(&out, d.cs, sizeof out, hipMemcpyDeviceToHost, st));
  PP_TRY(poll_stream(st));
  if (gwo) *gwo = out.gwo;
  if (objective) *objective = out.obj;
  return PP_OK;
}

int pp_marginal(int32_t n, int32_t m, const int64_t* demand,
                const int64_t* recompute_cost, const int64_t* fetch_cost,
                const uint8_t* target, int32_t h, int64_t* profit,
                int64_t* g_without_h) {
  g_err[0] = 0;
  return guarded([&]() -> int {
    if (!profit) return fail(PP_E_ARG, "null profit");
    if (m >= 1 && (h < 0 || h >= m)) return fail(PP_E_ARG, "h out of range");
    std::vector<int64_t> tmp(n > 0 ? n : 1);
    int64_t g = 0;
    PP_TRY(marginal_or_objective(n, m, demand, recompute_cost, fetch_cost,
                                 target, h, tmp.data(), &g, nullptr));
    std::copy(tmp.begin(), tmp.begin() + n, profit);
    if (g_without_h) *g_without_h = g;
    return PP_OK;
  });
}

int pp_objective(int32_t n, int32_t m, const int64_t* demand,
                 const int64_t* recompute_cost, const int64_t* fetch_cost,
                 const uint8_t* target, int64_t* objective) {
  g_err[0] = 0;
  return guarded([&]() -> int {
    if (!objective) return fail(PP_E_ARG, "null objective");
    int64_t v = 0;
    PP_TRY(marginal_or_objective(n, m, demand, recompute_cost, fetch_cost,
                                 target, 0, nullptr, nullptr, &v));
    *objective = v;
    return PP_OK;
  });
}

int pp_objective_device_noalloc(int32_t n, int32_t m, const int64_t* demand_dev,
                                const int64_t* recompute_dev, const int64_t* fetch_dev,
                                const uint8_t* target_dev, int64_t* objective,
                                void* hip_stream) {
  // no allocation of any kind on this path: errors go to the fixed buffer,
  // the kernels' partial sums to the library's per-GPU scratch array
  g_err[0] = 0;
  if (!demand_dev || !recompute_dev || !fetch_dev || !target_dev || !objective)
    return fail_c(PP_E_ARG, "null pointer argument");
  if (n < 1 || m < 1 || m > 255) return fail_c(PP_E_ARG, "need n >= 1 and 1 <= m <= 255");
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail_c(PP_E_DEVICE, "no current HIP device");
  void* scr = nullptr;
  hipError_t e = noalloc_scratch(dev, &scr);
  if (e != hipSuccess)
    return fail_c(PP_E_DEVICE, "looking up the scratch array (hipGetSymbolAddress) failed");
  NoAllocResult r{};
  e = launch_objective_noalloc(n, m, demand_dev, recompute_dev, fetch_dev, target_dev,
                               scr, &r, (hipStream_t)hip_stream);
  if (e != hipSuccess) return fail_c(PP_E_DEVICE, hipGetErrorString(e));
  if (r.bad) return fail_c(PP_E_RANGE, "negative demand, recompute cost or fetch cost");
  if (r.overflow)
    return fail_c(PP_E_OVERFLOW, "sum of demand * recompute cost exceeds INT64_MAX");
  *objective = r.objective;
  return PP_OK;
}

}  // extern "C"
