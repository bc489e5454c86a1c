// pp_internal.h -- shared declarations between the host driver (pp_host.cpp)
// and the gfx950 kernels (pp_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pp {

// Chains (one worker update each) handled by a single launch.
constexpr int kMaxChains = 64;
// Updates per launch in a speculative refinement sweep (all active starts
// together; a start's speculative updates beyond the first use spare slots).
constexpr int kSpecChains = 16;
// "no holder" marker of the top-1 holder state (workers are < 255).
constexpr uint8_t kNoHolder = 255;

// Per-step metadata of the DP sweep: four uint32 per padded step (see
// kDpBatch), encoded for a given cells-per-lane width C.  LDS rows hold
// 64*C int64 at a stride of dp_row_stride(C) bytes: H slot rows for far
// skip targets, the all-zero row, then dp_sink_rows(C) sink rows.
//   word 0: byte offset of the row that row i is stored to: its slot if it
//           is a far skip target (next(a) = i for some a < i-1), else sink
//           row (step mod dp_sink_rows(C)).
//   word 1: byte offset of the row read as the skip operand of the next
//           step (row i-1): the slot of next(i-1), or the zero row when
//           next(i-1) = n+1 or b_{i-1} is a leaf (whose skip operand, the
//           previous row, is in registers).
//   word 2: all ones when b_i is a leaf, else zero.
//   word 3: zero.
// Padded step 0 is a leaf.
constexpr int kMetaWords = 4;
// Sink rows (also the steps per gather of a stage's last cell column): 16
// at one cell per lane, 4 for wider rows to keep more stages resident.
// Slot reuse waits for the gather of a 16-step group, which covers both.
constexpr int kDpGatherMax = 16;
constexpr int dp_sink_rows(int cells) { return cells == 1 ? 16 : 4; }
// LDS row stride: 64*C int64 plus 8 bytes, so that lane 63 of consecutive
// rows falls in different banks.
constexpr int64_t dp_row_stride(int cells) { return (int64_t)cells * 64 * 8 + 8; }
constexpr int kMaxSlots = 254;
// Deep trees whose pending skip rows exceed the LDS slots spill the rows
// first read at least this many sweep batches after their store.
constexpr int kSpillGap = 3;
// The sweep runs steps in batches of kDpBatch; the step count is padded up
// to a multiple of it with leading dummy steps (leaf, profit 0), so step s
// of the tree is padded step s + pad, pad = nsteps - n.
constexpr int kDpBatch = 32;
// Rows per block of the backtrack's staged chain table (16 windows of 32).
constexpr int kCeBlock = 512;
// Exit row of a backtrack skip chain that leaves the last row: larger than
// any row of any super-window the walk can be in.
constexpr uint32_t kCeEnd = 0x7FFFFFFFu;  // = PP_BT_END of the public header

enum Mode : int32_t { kModeStandalone = 0, kModeGreedy = 1, kModeRefine = 2 };
// Profit of a worker update: the exact marginal of Eq. 7, or one of the
// requester-side comparator profits (Sec. IV-C safeguards).
enum GainsMode : int32_t {
  kGainsMarginal = 0,
  kGainsIndependent = 1,
  kGainsPopularity = 2,
  kGainsLocalDedup = 3
};

// Exact sums of real-valued objective terms.  A finite double x >= 0 is an
// integer number of units of 2^-1074; a sum of such terms is kept exactly as
// kExLimbs little-endian 32-bit limbs of that integer (2^2304 units, far
// above any sum of finite doubles), so it does not depend on the order of
// the additions.  Device accumulators are "lazy": 64-bit limbs that each
// collect 32-bit chunks and are carried once at the end.
constexpr int kExLimbs = 72;

// Where a term lands: x = mant * 2^pos units, split into 32-bit chunks at
// limbs limb, limb+1, limb+2 (chunk 2 < 2^21).  Returns false for x = 0.
__host__ __device__ inline bool ex_chunks(double x, int& limb, uint32_t& c0, uint32_t& c1,
                                          uint32_t& c2) {
  const uint64_t bits = __builtin_bit_cast(uint64_t, x);
  const int e = (int)(bits >> 52);
  uint64_t mant = bits & ((1ull << 52) - 1);
  int pos = 0;
  if (e > 0) {
    mant |= 1ull << 52;
    pos = e - 1;
  }
  if (mant == 0) return false;
  limb = pos >> 5;
  const int sh = pos & 31;
  const uint64_t lo = mant << sh;
  c0 = (uint32_t)lo;
  c1 = (uint32_t)(lo >> 32);
  c2 = sh ? (uint32_t)(mant >> (64 - sh)) : 0u;
  return true;
}

// a += x exactly (canonical limbs, carries propagated).
__host__ __device__ inline void ex_add_double(uint32_t* a, double x) {
  int limb;
  uint32_t c[3];
  if (!ex_chunks(x, limb, c[0], c[1], c[2])) return;
  uint64_t carry = 0;
  for (int q = limb; q < kExLimbs; ++q) {
    const uint64_t add = q - limb < 3 ? c[q - limb] : 0u;
    if (q - limb >= 3 && carry == 0) break;
    const uint64_t t = (uint64_t)a[q] + add + carry;
    a[q] = (uint32_t)t;
    carry = t >> 32;
  }
}

// -1, 0, 1 as a < b, a == b, a > b.
__host__ __device__ inline int ex_cmp(const uint32_t* a, const uint32_t* b) {
  for (int q = kExLimbs - 1; q >= 0; --q)
    if (a[q] != b[q]) return a[q] < b[q] ? -1 : 1;
  return 0;
}

// d = a - b for a >= b.
__host__ __device__ inline void ex_sub(uint32_t* d, const uint32_t* a, const uint32_t* b) {
  uint32_t borrow = 0;
  for (int q = 0; q < kExLimbs; ++q) {
    const uint64_t t = (uint64_t)a[q] - b[q] - borrow;
    d[q] = (uint32_t)t;
    borrow = (uint32_t)(t >> 63);
  }
}

// Bit pattern of the double nearest to a (ties to even; +inf beyond the
// largest finite double).
__host__ __device__ inline uint64_t ex_round_bits(const uint32_t* a) {
  int hi = kExLimbs - 1;
  while (hi >= 0 && a[hi] == 0) --hi;
  if (hi < 0) return 0;
  const int top = 32 * hi + 31 - __builtin_clz(a[hi]);  // highest set bit
  // bits [lo, top] of a as an integer (lo >= 0), at most 64 of them
  auto window = [&](int lo) -> uint64_t {
    uint64_t v = 0;
    for (int k = top; k >= lo; --k) v = v << 1 | ((a[k >> 5] >> (k & 31)) & 1u);
    return v;
  };
  if (top < 53) return window(0);  // exact: a denormal or the first binade
  uint64_t m = window(top - 52);   // 53 bits
  const int rb = top - 53;         // rounding bit
  const bool half = (a[rb >> 5] >> (rb & 31)) & 1u;
  bool sticky = false;
  for (int k = 0; k < (rb >> 5) && !sticky; ++k) sticky = a[k] != 0;
  if (!sticky) sticky = (a[rb >> 5] & ((1u << (rb & 31)) - 1u)) != 0;
  int t = top;
  if (half && (sticky || (m & 1))) {
    ++m;
    if (m == (1ull << 53)) {
      m >>= 1;
      ++t;
    }
  }
  const int64_t expo = (int64_t)t - 51;  // the value is m / 2^52 * 2^(t - 1074)
  if (expo >= 2047) return 0x7FFull << 52;
  return (uint64_t)expo << 52 | (m & ((1ull << 52) - 1));
}

// Scalars of one chain slot, updated on the device.
struct ChainState {
  int64_t dpval;     // D[1][k'] of the last DP sweep
  int64_t inc;       // sum of p_h over the incumbent T_h (refinement test)
  int64_t gwo;       // G(T_-h): objective with T_h emptied
  int64_t obj;       // objective of the chain's placement
  int32_t accept;    // last update adopted its DP result
  int32_t accepts;   // accepted refinement replacements so far
  int32_t status;    // nonzero: a device-side wait gave up
  // Real-valued refinement: the update was rejected before its walk (its
  // DP value is below the incumbent's value + eps by more than any
  // rounding of the two sums can account for), so no exact G is needed.
  int32_t rejected;
  int64_t wsum;      // real-valued: sum over (r, b) of Lambda * w (the
                     // scale of that rounding bound), double bits
  // Refinement updates whose inputs are unchanged: bit h of dirty is set
  // when another worker's replacement is adopted (its set may change) and
  // cleared when worker h's DP runs.
  // A refinement update of a clean worker would rebuild the same profits,
  // find the same set and reject it, so it is resolved as rejected without
  // the sweep (skip = 1 for the current update).
  int32_t skip;
  int32_t skips;           // updates resolved that way
  int64_t skipped_cells;   // their n * k' DP cells
  uint32_t dirty[8];       // one bit per worker (m <= 255)
};

// The chains of one launch, passed by value as a kernel argument.
struct ChainSet {
  int32_t count;
  int32_t slot[kMaxChains];    // state slot of the chain
  int32_t src[kMaxChains];     // slot whose placement k_gains reads (the
                               // chain's own slot, except for a speculative
                               // update computed in a spare slot)
  int32_t worker[kMaxChains];  // worker h being updated
  int32_t kprime[kMaxChains];  // min(k_h, n)
  int32_t base[kMaxChains + 1];  // DP: first block of each chain's stages
};

// Adoptions after a speculative refinement launch, one per start, passed
// by value as a kernel argument.
struct AdoptSet {
  int32_t count;
  int32_t slot[kMaxChains];    // the start's slot
  int32_t from[kMaxChains];    // spare slot of the accepted update, or -1
  int32_t worker[kMaxChains];  // its worker (from >= 0)
  uint32_t ran[kMaxChains][8]; // workers swept against the unchanged placement
};

// Device-resident problem and per-slot state of a context.
struct DevState {
  int32_t n, m;
  int32_t npad;             // n rounded up to a multiple of 64
  const int64_t* lam;       // [m][n]     demand, preorder positions
  const int64_t* w;         // [m][n]     recompute cost, preorder
  const int64_t* f;         // [m][m][n]  fetch cost [src][dst][pos]
  const int32_t* nextpos;   // [n]        0-based first position after subtree
  const uint32_t* ce;       // [nce][4]   backtrack skip chain of q in its
                            //            32-row window (bit per row), the
                            //            first row of that chain past the
                            //            window (kCeEnd: past the last
                            //            row), that row's own chain mask (0
                            //            for kCeEnd) and 0; nce = n rounded
                            //            up to kCeBlock, plus kCeBlock empty
                            //            rows (mask 0, exit kCeEnd)
  const uint32_t* meta;     // [nsteps][4] per-step DP metadata
  uint8_t* tgt;             // [slots][m][n] placement, preorder
  int64_t* v1;              // [slots][m][n] best holder saving
  int64_t* v2;              // [slots][m][n] best saving among other holders
  uint8_t* h1;              // [slots][m][n] holder giving v1
  int64_t* profit;          // [slots][n]    marginal profits p_h, preorder
  uint32_t* sel;            // [slots][npad/32] backtracked selection bitmap:
                            //   position q is bit q%32 of word q/32
  uint64_t* bits;           // [slots][stages][cells][npad] DP choice bits:
                            //   as uint32 words [2*npad] per (stage, cell),
                            //   word 64*b + l = lane l's cell over sweep
                            //   batch b, bit 31-u = step 32*b + u
  uint64_t* ring;           // [slots][stages][n][2] stage boundary values
  // Spilled skip rows (deep trees only; nspill = 0 otherwise): per sweep
  // batch b, sp_out[2e], sp_out[2e+1] for e in [sp_out_off[b],
  // sp_out_off[b+1]) = (temporary LDS slot, spill index) copied out once the
  // batch is done; sp_in likewise (restore LDS slot, spill index) copied in
  // when the batch is staged; spill = [slots][stages][nspill][64 * cells].
  const int32_t* sp_out_off;
  const int32_t* sp_out;
  const int32_t* sp_in_off;
  const int32_t* sp_in;
  uint64_t* spill;
  int32_t nspill;
  ChainState* cs;           // [slots]
  int32_t stages;           // stage stride of bits / ring
  int32_t cells;            // cells per lane of the DP sweep
  // Real-valued costs: every value array (lam, w, f, v1, v2, profit, the
  // ring and the ChainState values) then holds IEEE doubles, all finite
  // and non-negative, so their bit patterns order like the values.
  int32_t f64;
  double eps;               // refinement tolerance (real-valued costs)
  // Exact objective values (real-valued costs): gx[slot][0] = G of the
  // slot's placement, gx[slot][1] = G with the slot's last update adopted;
  // gxp = lazy per-block partial sums, [chain][gx_blocks][kExLimbs].
  uint32_t* gx;
  uint64_t* gxp;
  int32_t gx_blocks;
  // DP sweeps of at most this many stage blocks choose their waves' roles
  // by SIMD (0: every sweep); beyond four blocks per compute unit some
  // SIMDs carry two compute waves whatever the roles
  int32_t role_max_blocks;
};
// kernel arguments stay within the 4 KB that every launch path accepts
static_assert(sizeof(AdoptSet) + sizeof(DevState) <= 4096, "k_adopt arguments");
static_assert(sizeof(ChainSet) + sizeof(DevState) + 64 <= 4096, "ChainSet kernel arguments");

// Host-side launchers (pp_kernels.hip).  All enqueue on `st`.
hipError_t launch_gather(const int64_t* src, int64_t* dst, int32_t rows,
                         int32_t n, const int32_t* order, hipStream_t st);
// lam, w ([m][n]) and f ([m][m][n]) gathered to preorder in one launch
hipError_t launch_gather_inputs(const int64_t* lam, const int64_t* w, const int64_t* f,
                                int64_t* dlam, int64_t* dw, int64_t* df, int32_t m,
                                int32_t n, const int32_t* order, hipStream_t st);
hipError_t launch_gather_u8(const uint8_t* src, uint8_t* dst, int32_t rows,
                            int32_t n, const int32_t* order, hipStream_t st);
hipError_t launch_scatter_u8(const uint8_t* src, uint8_t* dst, int32_t rows,
                             int32_t n, const int32_t* order, hipStream_t st);
hipError_t launch_scatter_i64(const int64_t* src, int64_t* dst, int32_t n,
                              const int32_t* order, hipStream_t st);
// integer inputs, *nblocks (<= kValidateBlocks) blocks: partial[b] = block
// b's sum of lam*w (UINT64_MAX if it exceeds INT64_MAX), partial[nblocks +
// b] = 1 if block b saw a negative value, else 0
constexpr int kValidateBlocks = 1024;
hipError_t launch_validate(const int64_t* lam, const int64_t* w,
                           const int64_t* f, int32_t n, int32_t m,
                           uint64_t* partial, int32_t* nblocks, hipStream_t st);
// real-valued inputs, *nblocks (<= 2 kValidateBlocks) blocks: flags[b] = 1
// if block b saw a negative, NaN or infinite value, else 0
hipError_t launch_validate_f64(const double* lam, const double* w,
                               const double* f, int32_t n, int32_t m,
                               uint64_t* flags, int32_t* nblocks, hipStream_t st);
// Exact objective sums (real-valued costs): blocks per chain of k_gexact
// (128, or enough that no block sums more than 2^30 terms; m * n < 2^39).
constexpr int kGexactBlocks = 512;
int32_t gexact_blocks(int32_t n, int32_t m);
// mode kModeGreedy / kModeRefine: G of each update's placement (worker h's
// set replaced by its backtracked selection) and the acceptance decision;
// any other mode: G of each slot's own placement (gx[slot][0], cs.obj).
hipError_t launch_gexact(const ChainSet& set, const DevState& d, int mode,
                         hipStream_t st);
hipError_t launch_init_slots(const ChainSet& set, const DevState& d,
                             int clear_tgt, hipStream_t st);
hipError_t launch_holder_build(const ChainSet& set, const DevState& d,
                               hipStream_t st);
// may_skip: refinement updates, which resolve a clean worker's update
// without a sweep (see ChainState::dirty)
hipError_t launch_gains(const ChainSet& set, const DevState& d, hipStream_t st,
                        int gmode = kGainsMarginal, int may_skip = 0);
hipError_t launch_assemble(const ChainSet& set, const DevState& d, int32_t dst,
                           hipStream_t st);
hipError_t launch_requester_check(const int64_t* f, int32_t n, int32_t m,
                                  int32_t* mismatch, hipStream_t st);
// partial: at least 1024 exact sums (integer costs: 16 bytes each;
// real-valued: kExLimbs lazy 64-bit limbs each); *nblocks receives the count
hipError_t launch_mat_cost(const DevState& d, int32_t inc, int32_t prop,
                           void* partial, int32_t* nblocks, hipStream_t st);
hipError_t launch_dp(const ChainSet& set, const DevState& d, uint32_t epoch,
                     uint32_t spin_limit, int store_bits, int32_t slots_lds,
                     int fmax, hipStream_t st);
hipError_t launch_backtrack(const ChainSet& set, const DevState& d, int mode,
                            hipStream_t st);
// Speculative refinement: the updates of consecutive positions of one
// start run together in spare slots; per start, the first accepted one (in
// spare slot `from`, or none: from = -1) is adopted into the start's slot,
// whose stale-input marks lose the bits in `ran` (workers whose sweep ran
// against the unchanged placement).  One launch for every start.
hipError_t launch_adopt(const AdoptSet& set, const DevState& d, hipStream_t st);
// Greedy position 0: each chain adopts the standalone selection of its
// worker (row `worker` of sel0, [m][npad/32]) as its walk would have.
hipError_t launch_take_standalone(const ChainSet& set, const DevState& d,
                                 const uint32_t* sel0, hipStream_t st);
hipError_t launch_commit(const ChainSet& set, const DevState& d, int mode,
                         hipStream_t st);
hipError_t launch_objective(const ChainSet& set, const DevState& d,
                            hipStream_t st);

// Allocation-free objective (pp_objective_device_noalloc): the kernels' only
// device memory besides the caller's arrays is a file-scope array of
// kNoAllocScratchBytes per GPU (= PP_NOALLOC_SCRATCH_BYTES).
constexpr size_t kNoAllocScratchBytes = 40960;
constexpr int kNoAllocMaxDevices = 64;
struct NoAllocResult {
  int64_t objective;
  bool bad;       // a negative demand or cost
  bool overflow;  // sum of demand * recompute cost above INT64_MAX
};
// Device address of the scratch array on `device` (the current device),
// looked up once per device.
hipError_t noalloc_scratch(int device, void** ptr);
// Enqueue the objective kernels on `st`, copy the totals back and wait.
hipError_t launch_objective_noalloc(int32_t n, int32_t m, const int64_t* lam,
                                    const int64_t* w, const int64_t* f,
                                    const uint8_t* tgt, void* scr,
                                    NoAllocResult* out, hipStream_t st);

// Blocks of the DP sweep that can be resident at once for `cells` cells
// per lane and `slots_lds` stack slots (0 if unsupported).
int dp_resident_blocks(int cells, int32_t slots_lds, int device);
size_t dp_lds_bytes(int cells, int32_t slots_lds);

}  // namespace pp
