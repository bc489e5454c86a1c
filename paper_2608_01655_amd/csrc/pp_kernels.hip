// pp_kernels.hip -- gfx950 kernels of the PrefixPlace worker update.
//
// One worker update (Algorithm 1, PrefixPlace procedure) is four launches
// over every active chain (a chain is one start's current update, or one
// standalone solve):
//   k_gains      exact marginals p_h(b) (Eq. 7, Proposition 1) from the
//                top-2 holder state, plus the incumbent's value for the
//                strict-improvement test (Sec. IV-C)
//   k_dp<C>      the rooted-tree DP sweep of Eq. 9 (Theorem 1), pipelined
//                over the capacity axis: one stage (a compute wave and an
//                I/O wave) owns 64*C consecutive cells j; rows are swept
//                n..1 with no barrier
//   k_backtrack  the acceptance decision and the backtrack (Theorem 1's
//                "at most n states"), one wave per chain
//   k_commit     adopt T'_h and refresh the top-2 holder state on the chunks
//                whose membership changed
// plus the objective F_pair (Eq. 6) and small layout helpers.
//
// Values are int64 (integer costs) or, for real-valued costs, the bit
// patterns of finite non-negative doubles in the same 64-bit slots (the
// F64 template flag of k_dp, DevState::f64 elsewhere); indices are int32.

#include <algorithm>
#include <array>
#include <mutex>
#include <utility>
#include <vector>

#include "pp_internal.h"

namespace pp {

namespace {

constexpr int kWave = 64;

__device__ __forceinline__ int64_t imax(int64_t a, int64_t b) {
  return a > b ? a : b;
}

// Real-valued costs travel as the bit patterns of IEEE doubles.
__device__ __forceinline__ double as_f(int64_t v) { return __builtin_bit_cast(double, v); }
__device__ __forceinline__ int64_t as_i(double v) { return __builtin_bit_cast(int64_t, v); }
__device__ __forceinline__ double dpos(double v) { return v > 0.0 ? v : 0.0; }

// Eq. 5: saving of requester `r` when its copy of chunk `i` comes from
// holder `h` (fetch plane is [src][dst][pos]).  For real-valued costs the
// result is the bit pattern of a non-negative double, which compares like
// the value.
__device__ __forceinline__ int64_t saving(const DevState& d, int h, int r,
                                          int64_t i) {
  const int64_t wr = d.w[(int64_t)r * d.n + i];
  if (h == r) return wr;
  const int64_t fv = d.f[((int64_t)h * d.m + r) * d.n + i];
  if (d.f64) return as_i(dpos(as_f(wr) - as_f(fv)));
  return imax(wr - fv, 0);
}

// Top-2 holder state of chunk i for every requester, from slot s's
// placement: v1 = best saving over holders, h1 = its holder (lowest id on
// ties), v2 = best saving over holders other than h1 (0 if none).  The
// leave-one-out value of Eq. 7 is then v2 if h1 == h else v1.
__device__ void refresh_holders(const DevState& d, int64_t s, int64_t i) {
  const int64_t mn = (int64_t)d.m * d.n;
  const uint8_t* t = d.tgt + s * mn;
  for (int r = 0; r < d.m; ++r) {
    int64_t b1 = 0, b2 = 0;
    int hb = kNoHolder;
    for (int l = 0; l < d.m; ++l) {
      if (!t[(int64_t)l * d.n + i]) continue;
      const int64_t q = saving(d, l, r, i);
      if (hb == kNoHolder || q > b1) {
        b2 = (hb == kNoHolder) ? b2 : b1;
        b1 = q;
        hb = l;
      } else if (q > b2) {
        b2 = q;
      }
    }
    const int64_t o = s * mn + (int64_t)r * d.n + i;
    d.v1[o] = b1;
    d.v2[o] = b2;
    d.h1[o] = (uint8_t)hb;
  }
}


typedef int pp_int2 __attribute__((ext_vector_type(2)));
typedef int64_t pp_i64x2 __attribute__((ext_vector_type(2)));
typedef uint32_t pp_u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t pp_u32x3 __attribute__((ext_vector_type(3)));

__device__ __forceinline__ pp_int2 split64(int64_t v) {
  return __builtin_bit_cast(pp_int2, v);
}

__device__ __forceinline__ int64_t join64(pp_int2 v) {
  return __builtin_bit_cast(int64_t, v);
}


__device__ __forceinline__ uint64_t ld_agent(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void st_agent(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Sum over a 256-thread block, returned in thread 0.
__device__ int64_t block_sum(int64_t v) {
  __shared__ int64_t part[256 / kWave];
  for (int o = 32; o > 0; o >>= 1) v += __shfl_down(v, o, kWave);
  const int lane = threadIdx.x % kWave, wv = threadIdx.x / kWave;
  if (lane == 0) part[wv] = v;
  __syncthreads();
  int64_t t = 0;
  if (threadIdx.x == 0)
    for (int k = 0; k < (int)(blockDim.x / kWave); ++k) t += part[k];
  __syncthreads();
  return t;
}

// Sum of a double over a 256-thread block (any order), in thread 0.
__device__ double block_sum_f64(double v) {
  __shared__ double part[256 / kWave];
  for (int o = 32; o > 0; o >>= 1) v += __shfl_down(v, o, kWave);
  const int lane = threadIdx.x % kWave, wv = threadIdx.x / kWave;
  if (lane == 0) part[wv] = v;
  __syncthreads();
  double t = 0.0;
  if (threadIdx.x == 0)
    for (int k = 0; k < (int)(blockDim.x / kWave); ++k) t += part[k];
  __syncthreads();
  return t;
}

// Lazy exact accumulation of non-negative doubles into kExLimbs 64-bit
// limbs in LDS (each limb collects 32-bit chunks; the carries are taken
// when the block's partial is written).  A thread first adds its terms into
// a window of four limbs in registers, anchored one limb below its first
// term (the terms of one sum are mostly of similar size); a term outside the
// window goes to LDS at once, the window at the end (flush).
struct ExWindow {
  int base = -1;
  unsigned long long r0 = 0, r1 = 0, r2 = 0, r3 = 0;
};

__device__ __forceinline__ void ex_accumulate(unsigned long long* acc, ExWindow& win,
                                              double x) {
  int limb;
  uint32_t c0, c1, c2;
  if (!ex_chunks(x, limb, c0, c1, c2)) return;
  if (win.base < 0) win.base = limb > 0 ? limb - 1 : 0;
  const int o = limb - win.base;
  if (o == 0 || o == 1) {
    const unsigned long long a0 = c0, a1 = c1, a2 = c2;
    win.r0 += o == 0 ? a0 : 0ull;
    win.r1 += o == 0 ? a1 : a0;
    win.r2 += o == 0 ? a2 : a1;
    win.r3 += o == 0 ? 0ull : a2;
    return;
  }
  atomicAdd(acc + limb, (unsigned long long)c0);
  if (c1) atomicAdd(acc + limb + 1, (unsigned long long)c1);
  if (c2) atomicAdd(acc + limb + 2, (unsigned long long)c2);
}

__device__ __forceinline__ void ex_flush(unsigned long long* acc, const ExWindow& win) {
  if (win.base < 0) return;
  if (win.r0) atomicAdd(acc + win.base, win.r0);
  if (win.r1) atomicAdd(acc + win.base + 1, win.r1);
  if (win.r2) atomicAdd(acc + win.base + 2, win.r2);
  if (win.r3) atomicAdd(acc + win.base + 3, win.r3);
}

// ------------------------------------------------------------ helpers ---

// Values into preorder positions.  The bit pattern of -0.0 (INT64_MIN,
// never a valid integer input) becomes +0.0, so that real-valued inputs
// compare and order by their bit patterns.
__global__ void k_gather(const int64_t* __restrict__ src, int64_t* __restrict__ dst,
                         int32_t n, const int32_t* __restrict__ order) {
  const int64_t row = blockIdx.y;
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    const int64_t v = src[row * n + order[i]];
    dst[row * n + i] = v == INT64_MIN ? 0 : v;
  }
}

// The three inputs in one launch: rows [0, m) of lam, then of w, then the
// m*m rows of f.
__global__ void k_gather_inputs(const int64_t* __restrict__ lam, const int64_t* __restrict__ w,
                                const int64_t* __restrict__ f, int64_t* __restrict__ dlam,
                                int64_t* __restrict__ dw, int64_t* __restrict__ df, int32_t m,
                                int32_t n, const int32_t* __restrict__ order) {
  int64_t row = blockIdx.y;
  const int64_t* src = lam;
  int64_t* dst = dlam;
  if (row >= 2 * m) {
    row -= 2 * m;
    src = f;
    dst = df;
  } else if (row >= m) {
    row -= m;
    src = w;
    dst = dw;
  }
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    const int64_t v = src[row * n + order[i]];
    dst[row * n + i] = v == INT64_MIN ? 0 : v;
  }
}

__global__ void k_gather_u8(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                            int32_t n, const int32_t* __restrict__ order) {
  const int64_t row = blockIdx.y;
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[row * n + i] = src[row * n + order[i]];
}

__global__ void k_scatter_u8(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                             int32_t n, const int32_t* __restrict__ order) {
  const int64_t row = blockIdx.y;
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[row * n + order[i]] = src[row * n + i];
}

__global__ void k_scatter_i64(const int64_t* __restrict__ src, int64_t* __restrict__ dst,
                              int32_t n, const int32_t* __restrict__ order) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[order[i]] = src[i];
}

// Value checks of device-resident inputs: negatives are flagged, and each
// block's sum of lam*w is returned (saturated to UINT64_MAX on overflow) for
// the host to add exactly.
__global__ void k_validate(const int64_t* __restrict__ lam, const int64_t* __restrict__ w,
                           const int64_t* __restrict__ f, int64_t mn, int64_t mmn,
                           uint64_t* partial) {
  uint64_t acc = 0;
  bool ovf = false, bad = false;
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < mmn;
       x += (int64_t)gridDim.x * blockDim.x) {
    if (f[x] < 0) bad = true;
    if (x < mn) {
      const int64_t a = lam[x], b = w[x];
      if (a < 0 || b < 0) {
        bad = true;
        continue;
      }
      uint64_t prod;
      if (__builtin_mul_overflow((uint64_t)a, (uint64_t)b, &prod) ||
          prod > (uint64_t)INT64_MAX || acc + prod > (uint64_t)INT64_MAX)
        ovf = true;
      else
        acc += prod;
    }
  }
  // this block's flag: partial[gridDim.x + block] (every block writes its
  // own, so nothing needs clearing first)
  const int any_bad = __syncthreads_or(bad ? 1 : 0);
  if (threadIdx.x == 0) partial[gridDim.x + blockIdx.x] = any_bad ? 1 : 0;
  // block sum with saturation: each term is <= INT64_MAX, so two fit u64
  __shared__ uint64_t part[256];
  part[threadIdx.x] = ovf ? UINT64_MAX : acc;
  __syncthreads();
  for (int o = blockDim.x / 2; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) {
      const uint64_t a = part[threadIdx.x], b = part[threadIdx.x + o];
      part[threadIdx.x] = (a > (uint64_t)INT64_MAX || b > (uint64_t)INT64_MAX ||
                           a + b > (uint64_t)INT64_MAX) ? UINT64_MAX : a + b;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) partial[blockIdx.x] = part[0];
}

// Reset chain slots: empty placement (optional), zero holder state and
// chain scalars.
// Real-valued inputs: any negative, NaN or infinite value sets *bad.
__global__ void k_validate_f64(const double* __restrict__ lam,
                               const double* __restrict__ w,
                               const double* __restrict__ f, int64_t mn,
                               int64_t mmn, uint64_t* flags) {
  bool b = false;
  const int64_t step = (int64_t)gridDim.x * blockDim.x;
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < mmn; x += step) {
    const double fv = f[x];
    b |= !(fv >= 0.0 && fv <= 1.7976931348623157e308);
    if (x < mn) {
      const double a = lam[x], c = w[x];
      b |= !(a >= 0.0 && a <= 1.7976931348623157e308);
      b |= !(c >= 0.0 && c <= 1.7976931348623157e308);
    }
  }
  // this block's flag (every block writes its own: nothing to clear first)
  const int any = __syncthreads_or(b ? 1 : 0);
  if (threadIdx.x == 0) flags[blockIdx.x] = any ? 1 : 0;
}

__global__ void k_init_slots(ChainSet set, DevState d, int clear_tgt) {
  const int ci = blockIdx.y;
  const int64_t s = set.slot[ci];
  const int64_t mn = (int64_t)d.m * d.n;
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < mn;
       x += (int64_t)gridDim.x * blockDim.x) {
    if (clear_tgt) d.tgt[s * mn + x] = 0;
    d.v1[s * mn + x] = 0;
    d.v2[s * mn + x] = 0;
    d.h1[s * mn + x] = kNoHolder;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    ChainState z = {};
    d.cs[s] = z;
  }
  if (d.gx && clear_tgt && blockIdx.x == 0)  // G of the empty placement
    for (int q = threadIdx.x; q < 2 * kExLimbs; q += blockDim.x) d.gx[s * 2 * kExLimbs + q] = 0;
}

__global__ void k_holder_build(ChainSet set, DevState d) {
  const int ci = blockIdx.y;
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i < d.n) refresh_holders(d, set.slot[ci], i);
}

// ------------------------------------------------------------- gains ----

// p_h(b) = sum_m Lambda_m(b) [q_{m<-h}(b) - v_m^{(-h)}(b)]_+  (Eq. 7) for
// every preorder position, written to the chain's profit row; also the
// incumbent's value sum_{b in T_h} p_h(b) and G(T_-h) = sum Lambda v^{(-h)}.
// The comparator profits of the requester-side safeguards (Sec. IV-C) use
// the same path: Independent p = Lambda_h w_h, Popularity p = Lambda_h,
// LocalDedup p = a_h(b) + 1{b not held by another worker} Lambda_h
// [w_h - f_h]_+ (a_h = Lambda_h min(w_h, f_h), Eq. 2; f_h the common fetch
// cost of requester h; with one worker p = Lambda_h w_h).
__global__ void __launch_bounds__(256) k_gains(ChainSet set, DevState d, int gmode,
                                               int may_skip) {
  const int ci = blockIdx.y;
  const int64_t s = set.slot[ci];   // the update's own state: profit, sums
  const int64_t ps = set.src[ci];   // the placement it is computed against
  const int h = set.worker[ci];
  const int64_t n = d.n;
  const int64_t mn = (int64_t)d.m * n;
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  {
    // a refinement update of a worker whose inputs have not changed since
    // its last sweep: resolved as rejected, no gains, sweep or walk
    const bool clean = may_skip && gmode == kGainsMarginal &&
                       ((d.cs[ps].dirty[h >> 5] >> (h & 31)) & 1u) == 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      d.cs[s].skip = clean ? 1 : 0;
      if (clean) {
        d.cs[s].skips += 1;
        d.cs[s].skipped_cells += n * set.kprime[ci];
      }
    }
    if (clean) return;
  }
  if (gmode != kGainsMarginal && d.f64) {
    // the comparator profits on doubles, with the integer path's formulas
    if (i >= n) return;
    const double L = as_f(d.lam[(int64_t)h * n + i]), Wv = as_f(d.w[(int64_t)h * n + i]);
    double p;
    if (gmode == kGainsIndependent) {
      p = L * Wv;
    } else if (gmode == kGainsPopularity) {
      p = L;
    } else if (d.m == 1) {
      p = L * Wv;
    } else {
      const int src = h == 0 ? 1 : 0;
      const double F = as_f(d.f[((int64_t)src * d.m + h) * n + i]);
      bool covered = false;
      for (int l = 0; l < d.m; ++l)
        if (l != h && d.tgt[ps * mn + (int64_t)l * n + i]) covered = true;
      const double a = L * (Wv < F ? Wv : F);
      const double own = L * dpos(Wv - F);
      p = covered ? a : a + own;
    }
    d.profit[s * n + i] = as_i(p);
    return;
  }
  if (gmode != kGainsMarginal) {
    if (i >= n) return;
    const int64_t L = d.lam[(int64_t)h * n + i], Wv = d.w[(int64_t)h * n + i];
    int64_t p;
    if (gmode == kGainsIndependent) {
      p = L * Wv;
    } else if (gmode == kGainsPopularity) {
      p = L;
    } else if (d.m == 1) {
      p = L * Wv;
    } else {
      const int src = h == 0 ? 1 : 0;
      const int64_t F = d.f[((int64_t)src * d.m + h) * n + i];
      bool covered = false;
      for (int l = 0; l < d.m; ++l)
        if (l != h && d.tgt[ps * mn + (int64_t)l * n + i]) covered = true;
      const int64_t a = L * (Wv < F ? Wv : F);
      p = covered ? a : a + L * imax(Wv - F, 0);
    }
    d.profit[s * n + i] = p;
    return;
  }
  if (d.f64) {
    // Eq. 7 on doubles: requester terms added in increasing r, each product
    // rounded on its own.  The acceptance test evaluates G exactly (in
    // k_gexact); the incumbent's value sum_{b in T_h} p_h(b) and the scale
    // sum Lambda * w summed here (in any order) only let k_backtrack reject
    // an update early when no rounding could make it acceptable.
    double p = 0.0, wl = 0.0;
    bool in_th = false;
    if (i < n) {
      for (int r = 0; r < d.m; ++r) {
        const int64_t o = ps * mn + (int64_t)r * n + i;
        const double vmh = as_f((d.h1[o] == h) ? d.v2[o] : d.v1[o]);
        const double L = as_f(d.lam[(int64_t)r * n + i]);
        const double term = L * dpos(as_f(saving(d, h, r, i)) - vmh);
        p = p + term;
        wl = wl + L * as_f(d.w[(int64_t)r * n + i]);
      }
      d.profit[s * n + i] = as_i(p);
      in_th = d.tgt[ps * mn + (int64_t)h * n + i] != 0;
    }
    const double sh = block_sum_f64(in_th ? p : 0.0);
    const double sw = block_sum_f64(wl);
    if (threadIdx.x == 0) {
      if (sh != 0.0) atomicAdd((double*)&d.cs[s].inc, sh);
      if (sw != 0.0) atomicAdd((double*)&d.cs[s].wsum, sw);
    }
    return;
  }
  int64_t p = 0, g = 0, held = 0;
  if (i < n) {
    for (int r = 0; r < d.m; ++r) {
      const int64_t o = ps * mn + (int64_t)r * n + i;
      const int64_t vmh = (d.h1[o] == h) ? d.v2[o] : d.v1[o];
      const int64_t L = d.lam[(int64_t)r * n + i];
      p += L * imax(saving(d, h, r, i) - vmh, 0);
      g += L * vmh;
    }
    d.profit[s * n + i] = p;
    held = d.tgt[ps * mn + (int64_t)h * n + i] ? p : 0;
  }
  const int64_t sh = block_sum(held);
  const int64_t sg = block_sum(g);
  if (threadIdx.x == 0) {
    if (sh) atomicAdd((unsigned long long*)&d.cs[s].inc, (unsigned long long)sh);
    if (sg) atomicAdd((unsigned long long*)&d.cs[s].gwo, (unsigned long long)sg);
  }
}

// ------------------------------------------------------------ DP sweep --

// acc * 2 + (t > sk): the lane's choice bit of this step shifted into its
// 32-step word (the compare's lane mask is the add's carry-in).  F64: the
// values are doubles.
template <bool F64>
__device__ __forceinline__ uint32_t shift_in_gt(int64_t t, int64_t sk,
                                                uint32_t acc) {
  uint32_t r;
  if constexpr (F64)
    asm("v_cmp_gt_f64 vcc, %1, %2\n\tv_addc_co_u32_e32 %0, vcc, %3, %3, vcc"
        : "=v"(r)
        : "v"(as_f(t)), "v"(as_f(sk)), "v"(acc)
        : "vcc");
  else
    asm("v_cmp_gt_i64 vcc, %1, %2\n\tv_addc_co_u32_e32 %0, vcc, %3, %3, vcc"
        : "=v"(r)
        : "v"(t), "v"(sk), "v"(acc)
        : "vcc");
  return r;
}

// a + b on integers, or on the doubles the bit patterns encode
template <bool F64>
__device__ __forceinline__ int64_t vadd(int64_t a, int64_t b) {
  if constexpr (F64)
    return as_i(as_f(a) + as_f(b));
  else
    return a + b;
}

// Take operands of a DP row: lanes 1..63 get r + v of lane l-1 (a 64-bit
// add whose first operand is shifted in by DPP wave_shr:1); lane 0, whose
// shifted operand is zero (bound_ctrl), gets r.  A DPP read of a VGPR needs
// two wait states after the VALU write of that VGPR: take_after_bit puts
// the previous step's choice bit (t_prev > sk_prev, shifted into acc; two
// instructions) in front of the shift, take_first pads with s_nop.
__device__ __forceinline__ int64_t take_after_bit_i64(int64_t r, int64_t v, int64_t t_prev,
                                                      int64_t sk_prev, uint32_t& acc) {
  const pp_int2 rv = split64(r), vv = split64(v);
  pp_int2 t;
  asm("v_cmp_gt_i64 vcc, %3, %4\n\t"
      "v_addc_co_u32_e32 %0, vcc, %0, %0, vcc\n\t"
      "v_add_co_u32_dpp %1, vcc, %5, %7 wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
      "v_addc_co_u32_dpp %2, vcc, %6, %8, vcc wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
      : "+v"(acc), "=&v"(t.x), "=v"(t.y)
      : "v"(t_prev), "v"(sk_prev), "v"(vv.x), "v"(vv.y), "v"(rv.x), "v"(rv.y)
      : "vcc");
  return join64(t);
}

__device__ __forceinline__ int64_t take_first_i64(int64_t r, int64_t v) {
  const pp_int2 rv = split64(r), vv = split64(v);
  pp_int2 t;
  asm("s_nop 1\n\t"
      "v_add_co_u32_dpp %0, vcc, %2, %4 wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
      "v_addc_co_u32_dpp %1, vcc, %3, %5, vcc wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
      : "=&v"(t.x), "=v"(t.y)
      : "v"(vv.x), "v"(vv.y), "v"(rv.x), "v"(rv.y)
      : "vcc");
  return join64(t);
}

// Real-valued costs: v_add_f64 has no DPP form, so the left lane's 64-bit
// value is moved across first (two DPP moves, wave_shr:1, zero for lane 0
// by bound_ctrl) and added as doubles; lane 0 then gets r + 0.0 = r (r is a
// non-negative double).  The compiler inserts the DPP wait states.
__device__ __forceinline__ int64_t take_f64(int64_t r, int64_t v) {
  const pp_int2 vv = split64(v);
  pp_int2 sh;
  sh.x = __builtin_amdgcn_update_dpp(0, vv.x, 0x138, 0xf, 0xf, true);
  sh.y = __builtin_amdgcn_update_dpp(0, vv.y, 0x138, 0xf, 0xf, true);
  return as_i(as_f(r) + as_f(join64(sh)));
}

// LDS byte address of a row cell: base + 8 * (low or high 16-bit half of w),
// one v_mad_u32_u16 (op_sel picks the high half).
__device__ __forceinline__ uint32_t lds_row_lo(uint32_t w, uint32_t base) {
  uint32_t a;
  asm("v_mad_u32_u16 %0, %1, 8, %2" : "=v"(a) : "v"(w), "v"(base));
  return a;
}

__device__ __forceinline__ uint32_t lds_row_hi(uint32_t w, uint32_t base) {
  uint32_t a;
  asm("v_mad_u32_u16 %0, %1, 8, %2 op_sel:[1,0,0,0]" : "=v"(a) : "v"(w), "v"(base));
  return a;
}

typedef __attribute__((address_space(3))) int64_t lds_i64;

__device__ __forceinline__ lds_i64* lds_at(uint32_t a) { return (lds_i64*)(size_t)a; }

// Maximum of two non-negative int64 values below 2^62 with one v_max_f64:
// such bit patterns are finite non-negative doubles (denormals included,
// which the kernel's FP64 mode preserves), and IEEE 754 orders them exactly
// as the integers they encode, so the result is the larger integer.
__device__ __forceinline__ int64_t max_nonneg_f64(int64_t a, int64_t b) {
  double r;
  asm("v_max_f64 %0, %1, %2"
      : "=v"(r)
      : "v"(__builtin_bit_cast(double, a)), "v"(__builtin_bit_cast(double, b)));
  return __builtin_bit_cast(int64_t, r);
}

// Eq. 9, rows i = n..1, cells j = 1..k':
//   D[i][j] = max(D[next(i)][j], p(b_i) + D[i+1][j-1]),  D[n+1][*] = 0,
//   D[*][0] = 0;  choice bit = (take > skip)  (ties keep the skip branch).
//
// Layout: a chain's k' cells are split over G stages; stage g is a block
// of two waves owning cells j = g*64*C + l*C + c + 1 (lane l, c < C) of
// the compute wave.  Row i+1 stays in its registers.  The take operand
// p + D[i+1][j-1] is one add whose D operand comes from the left neighbour
// lane by DPP; lane 0's comes from stage g-1, whose last cell of every row
// is published through a per-step ring in global memory, and is added to p
// by the other wave, which does all global-memory traffic of the stage.
// Ring words carry a launch tag in their high half (relaxed agent-scope
// atomics, no fences): a consumer validates each word by its tag.  A stage
// loads its input two batches ahead, so in steady state it runs two
// batches behind its producer and finds the words there.
//
// Rows that a later row skips to (next(a) = i for some non-leaf a, i !=
// n+1) are stored to an LDS slot at their own step, other rows to one of a
// few sink rows (step mod their count), so the store needs no branch.
// Right after its store a step reads the skip operand of the step two
// ahead (a slot, or the all-zero row): that row is produced at this step at
// the latest.  A leaf's skip operand is the previous row, in registers,
// chosen per step by a uniform lane mask from the metadata.  After every
// group of sink-row-count steps the stage gathers its last cell column of
// those steps from the rows they were stored to (a slot is reused only
// after that gather) for the ring in global memory.
//
// Steps run in batches of kBatch, unrolled at compile time; the step count
// is padded up to a multiple of kBatch with leading dummy steps (profit 0,
// leaf, rows stay all-zero).  Per batch the I/O wave stages each step's
// record -- profit (plus the boundary value for lane 0), the packed row
// offsets and the leaf mask -- in LDS, read back by the compute wave with
// one load per step.  The waves hand batches over through two LDS counters
// (no barrier in the batch loop).  Each lane shifts its cells' choice bits
// into one 32-bit word per cell per batch (bit 31-u = step u), stored with
// one coalesced store per cell; the stage ring output also leaves with one
// store per batch.  No per-row launch, barrier or HBM row traffic.
constexpr int kBatch = kDpBatch;

// A step's record in two 16-byte views: lanes 1..63 read view 0, lane 0
// reads view 1, with one LDS read per step.
struct __attribute__((aligned(16))) StepView {
  int64_t r;      // view 0: the profit p of the step's node; view 1: p plus
                  // D[i+1][first cell - 1] from stage g-1 (0 for stage 0),
                  // lane 0's take operand
  uint32_t rows;  // low half: byte offset of the row this step is stored
                  // to, high half: of the next step's skip row; both / 8
  uint32_t leaf;  // all ones when the step's node is a leaf, else zero
};

template <int U>
using IC = std::integral_constant<int, U>;

template <class F, int... U>
__device__ __forceinline__ void unroll_steps(F&& f, std::integer_sequence<int, U...>) {
  (f(IC<U>{}), ...);
}

// Stage-ring values of a batch in the LDS output buffer: one per lane at
// one cell per lane (lanes < kBatch carry a step's; every lane stores, see
// k_dp), else one per step.
template <int C>
constexpr int dp_outv_stride() {
  return C == 1 ? kWave : kBatch;
}

// LDS bytes of the sweep's control area: two record buffers, two output
// buffers (stage-ring values and choice words of a batch) and four flag
// words (the two hand-off counters and the waves' role decision).
template <int C>
constexpr size_t dp_ctl_bytes() {
  return 2 * (kBatch + 1) * 2 * sizeof(StepView) + 2 * dp_outv_stride<C>() * sizeof(int64_t) +
         2 * C * kWave * sizeof(uint32_t) + 16;
}

// Compute waves per SIMD: bit s of g_simd_claims[cu] is set while a sweep's
// compute wave runs on SIMD s of compute unit cu (a key made of the XCD,
// shader engine, shader array and CU ids; each field is masked to its
// width, so every key indexes the table).  One table per device, zero at
// load; every wave that sets a bit clears it before it exits.
constexpr int kSimdClaimKeys = 1 << 12;
__device__ uint32_t g_simd_claims[kSimdClaimKeys];
constexpr int kHwIdReg = (31 << 11) | 4;    // s_getreg: HW_ID, 32 bits
constexpr int kXccIdReg = (31 << 11) | 20;  // s_getreg: XCC_ID, 32 bits

template <int C, bool FMAX, bool F64>
__global__ void __launch_bounds__(2 * kWave)
k_dp(ChainSet set, DevState d, uint32_t epoch, uint32_t spin_limit,
     int store_bits, int32_t slots) {
  extern __shared__ int64_t lds[];
  constexpr int kStride = (int)dp_row_stride(C);  // bytes per LDS row
  constexpr int kProd = dp_sink_rows(C);  // steps per gather of the last column
  static_assert(kBatch % kProd == 0 && kProd <= kDpGatherMax, "gather groups");
  // control area first (small immediate offsets), then the rows: the slots,
  // the zero row and the sink rows
  StepView* recs = (StepView*)lds;                             // [2][kBatch + 1][2]
  constexpr int kOutv = dp_outv_stride<C>();
  int64_t* outv = (int64_t*)(recs + 2 * (kBatch + 1) * 2);     // [2][kOutv]
  uint32_t* outb = (uint32_t*)(outv + 2 * kOutv);              // [2][C][64]
  // Hand-off between the waves through two LDS counters: sync[kStaged] =
  // batches whose records are staged (-1: the I/O wave gave up), sync[kDone]
  // = batches the compute wave has finished (their outputs are in LDS and
  // their record buffer is free; -1: it gave up).  A wave's LDS operations
  // execute in order, so LDS data written before a counter update is in
  // place for a wave that reads the counter and then the data; compiler
  // fences keep that program order, and no wave waits on the LDS counter.
  int* sync = (int*)(outb + 2 * C * kWave);
  constexpr int kStaged = 0, kDone = 1, kRole = 2;
  // bound on the polls of one LDS wait (the partner wave's own waits are
  // bounded, so this is reached only if the hand-off itself breaks)
  constexpr uint32_t kLdsSpins = 1u << 24;
  auto sync_load = [&](int t) {
    return __hip_atomic_load(sync + t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  };
  auto sync_get = [&](int t) { return __builtin_amdgcn_readfirstlane(sync_load(t)); };
  auto sync_set = [&](int t, int v) {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    if (threadIdx.x % kWave == 0)
      __hip_atomic_store(sync + t, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  };
  char* rows = (char*)lds + dp_ctl_bytes<C>();
  // one wave computes the sweep (role 0); the other does every global-memory
  // access of the batch loop (role 1), so the compute wave never waits on a
  // memory counter
  const int hw_wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  const int lane = threadIdx.x % kWave;
  char* lane_bytes = rows + lane * 8;
  const int blk = blockIdx.x;
  if (blk >= set.base[set.count]) return;
  int ci = 0;
  while (ci + 1 < set.count && set.base[ci + 1] <= blk) ++ci;
  const int64_t slot = set.slot[ci];
  if (d.cs[slot].skip) return;  // the update is resolved without a sweep
  const int kp = set.kprime[ci];
  const int g = blk - set.base[ci];
  const int G = set.base[ci + 1] - set.base[ci];
  const int n = d.n;
  const int nsteps = (n + kBatch - 1) / kBatch * kBatch;
  const int nb = nsteps / kBatch;
  const int pad = nsteps - n;  // leading dummy steps
  // Barrier between the two waves.  Only LDS is exchanged through it, so
  // the fences order LDS alone.
  auto barrier = [&]() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
  };
  // Roles.  The hardware puts the block's two waves on two SIMDs of its
  // compute unit; with three or more blocks on one compute unit, two
  // compute waves can share a SIMD, which runs both at about half pace and
  // holds back both chains.  So the compute role goes to a wave whose SIMD
  // no other compute wave has claimed: wave 0 if its SIMD is free, else
  // wave 1 if its SIMD is, else wave 0 without a claim.  (Claiming both at
  // once and giving one back was slower: the claim a block gives back can
  // turn another block away from a SIMD that stays free.)  Launches of more
  // than d.role_max_blocks blocks skip the claims: some SIMD carries two
  // compute waves there whatever the roles.
  const uint32_t hw_id = __builtin_amdgcn_s_getreg(kHwIdReg);
  const uint32_t cu_key = ((__builtin_amdgcn_s_getreg(kXccIdReg) & 0xFu) << 8) |
                          (((hw_id >> 13) & 7u) << 5) | (((hw_id >> 12) & 1u) << 4) |
                          ((hw_id >> 8) & 0xFu);
  const uint32_t simd_bit = 1u << ((hw_id >> 4) & 3u);
  uint32_t* const claim = g_simd_claims + cu_key;
  auto try_claim = [&]() {
    uint32_t old = 0;
    if (lane == 0) old = atomicOr(claim, simd_bit);
    return (__builtin_amdgcn_readfirstlane((int)old) & (int)simd_bit) == 0;
  };
  const bool roles = d.role_max_blocks == 0 || set.base[set.count] <= d.role_max_blocks;
  bool claimed = false;
  if (hw_wave == 0) {
    if (roles) claimed = try_claim();
    if (lane == 0) sync[kRole] = (claimed || !roles) ? 0 : -1;
  }
  barrier();
  if (hw_wave == 1 && __builtin_amdgcn_readfirstlane(sync_load(kRole)) < 0) {
    claimed = try_claim();
    if (lane == 0) sync[kRole] = claimed ? 1 : 0;
  }
  barrier();
  const int wave =
      hw_wave == __builtin_amdgcn_readfirstlane(sync_load(kRole)) ? 0 : 1;
  auto release_claim = [&]() {
    if (claimed && lane == 0) atomicAnd(claim, ~simd_bit);
  };

  if (wave == 1) {
    // ---------------------------------------------------------- I/O wave
    const int64_t stride = (int64_t)d.npad;  // steps per stage row of the ring
    const int64_t cstride = 2 * stride;      // choice words per (stage, cell)
    const int64_t* __restrict__ prof = d.profit + slot * n;
    const uint4* __restrict__ meta = (const uint4*)d.meta;  // [nsteps], padded
    uint32_t* bits = (uint32_t*)d.bits + (slot * d.stages + g) * (int64_t)C * cstride;
    uint64_t* ring_out = d.ring + (slot * d.stages + g) * stride * 2;
    const uint64_t* ring_in = (g > 0) ? ring_out - stride * 2 : nullptr;
    const uint64_t tag = (uint64_t)epoch << 32;
    const bool produce = g + 1 < G;
    // ring input of the batch at s0: lane u <= kBatch <- entry s0+u-1 (lane
    // kBatch: the following batch's first step, in the same producer batch)
    auto ring_load = [&](int s0, uint64_t& w0, uint64_t& w1) {
      const int e = s0 - 1 + lane;
      w0 = tag;
      w1 = tag;
      if (ring_in && lane <= kBatch && e >= 0 && s0 < nsteps) {
        w0 = ld_agent(ring_in + 2 * (int64_t)e);
        w1 = ld_agent(ring_in + 2 * (int64_t)e + 1);
      }
    };
    auto ring_ok = [&](uint64_t w0, uint64_t w1) {
      const bool ok = (w0 & 0xFFFFFFFF00000000ull) == tag &&
                      (w1 & 0xFFFFFFFF00000000ull) == tag;
      return __builtin_amdgcn_ballot_w64(ok) == ~0ull;
    };
    uint32_t spins = 0;
    auto ring_wait = [&](int s0, uint64_t& w0, uint64_t& w1) -> bool {
      while (!ring_ok(w0, w1)) {
        if (++spins > spin_limit) return false;
        __builtin_amdgcn_s_sleep(2);
        ring_load(s0, w0, w1);
      }
      return true;
    };
    // profit of padded step t (0 for the leading dummy steps and past the
    // end)
    auto profit_at = [&](int t) -> int64_t {
      const int s = t - pad;
      return (lane <= kBatch && s >= 0 && s < n) ? prof[n - 1 - s] : 0;
    };
    // lane kBatch carries the first step of the following batch: a batch's
    // record kBatch is the following batch's record 0
    auto meta_at = [&](int t) -> uint4 {
      return (lane <= kBatch && t < nsteps) ? meta[t] : make_uint4(0u, 0u, 0u, 0u);
    };
    // Spilled skip rows (deep trees): this stage's rows in device memory,
    // one 64*C-value row per spill index, lane l holding cells l + 64c.
    const bool spilling = d.nspill > 0;
    uint64_t* spill_rows =
        spilling ? d.spill + (slot * d.stages + g) * (int64_t)d.nspill * (kWave * C) : nullptr;
    auto lds_cell = [&](int32_t row_slot, int c) -> int64_t* {
      return (int64_t*)(rows + (int64_t)row_slot * kStride + c * kWave * 8 + lane * 8);
    };
    // copy-in of the rows that batch b reads from a restore slot, before
    // its records are published (a lane's relaxed agent-scope accesses to
    // one address stay in program order, so it reads what it spilled)
    auto spill_in = [&](int b) {
      for (int32_t e = d.sp_in_off[b]; e < d.sp_in_off[b + 1]; ++e) {
        const int32_t rs = d.sp_in[2 * e], x = d.sp_in[2 * e + 1];
#pragma unroll
        for (int c = 0; c < C; ++c)
          *lds_cell(rs, c) =
              (int64_t)ld_agent(spill_rows + (int64_t)x * (kWave * C) + c * kWave + lane);
      }
    };
    // copy-out of the spilled rows batch b stored to temporary slots, once
    // the batch is done (before the batch after next is staged)
    auto spill_out = [&](int b) {
      for (int32_t e = d.sp_out_off[b]; e < d.sp_out_off[b + 1]; ++e) {
        const int32_t ts = d.sp_out[2 * e], x = d.sp_out[2 * e + 1];
#pragma unroll
        for (int c = 0; c < C; ++c)
          st_agent(spill_rows + (int64_t)x * (kWave * C) + c * kWave + lane,
                   (uint64_t)*lds_cell(ts, c));
      }
    };
    auto stage = [&](int b, int64_t pv, uint64_t w0, uint64_t w1, uint4 mv) {
      if (spilling) spill_in(b);
      if (lane <= kBatch) {
        const int64_t bnd = (int64_t)((w1 << 32) | (w0 & 0xFFFFFFFFull));
        StepView v;
        v.r = pv;
        v.rows = (mv.x >> 3) | ((mv.y >> 3) << 16);
        v.leaf = mv.z;
        StepView* dst = recs + ((b % 2) * (kBatch + 1) + lane) * 2;
        dst[0] = v;
        v.r = vadd<F64>(pv, bnd);  // no overflow: a feasible set's value
        dst[1] = v;
      }
    };
    // the outputs of batch b, in LDS once sync[kDone] > b
    auto store_out = [&](int b) {
      if (store_bits) {
        const int64_t wi = (int64_t)b * kWave + lane;
#pragma unroll
        for (int c = 0; c < C; ++c)
          bits[c * cstride + wi] = outb[((b % 2) * C + c) * kWave + lane];
      }
      if (produce && lane < kBatch) {
        const uint64_t bo = (uint64_t)outv[(b % 2) * kOutv + lane];
        const int idx = b * kBatch + lane;
        st_agent(ring_out + 2 * (int64_t)idx, tag | (bo & 0xFFFFFFFFull));
        st_agent(ring_out + 2 * (int64_t)idx + 1, tag | (bo >> 32));
      }
      if (spilling) spill_out(b);
    };
    if (lane == 0) sync[kDone] = 0;
    bool ok;
    {
      // the records' other inputs first: they do not wait on the ring
      const int64_t p0 = profit_at(lane);
      const uint4 m0 = meta_at(lane);
      uint64_t w0, w1;
      ring_load(0, w0, w1);
      ok = ring_wait(0, w0, w1);
      stage(0, p0, w0, w1, m0);
    }
    // inputs of batch b+1, loaded during batch b-1 (ring words two batches
    // ahead; the validation waits only on loads)
    uint64_t a0, a1;
    ring_load(kBatch, a0, a1);
    int64_t pa = profit_at(kBatch + lane);
    uint4 ma = meta_at(kBatch + lane);
    if (lane == 0) sync[kStaged] = ok ? 1 : -1;
    barrier();
    // While the compute wave runs: publish each finished batch's outputs at
    // once (the next stage waits on them), and stage the next batch once
    // the compute wave has released its record buffer (batch nstage-2 done)
    // and its ring input (loaded when the previous batch was staged) is valid.
    int nstore = 0, nstage = 1;
    uint32_t idle = 0;
    while (ok && nstore < nb) {
      const int done = sync_get(kDone);
      if (done < 0) {
        ok = false;
        break;
      }
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      bool progress = false;
      if (done > nstore) {
        store_out(nstore);
        ++nstore;
        progress = true;
      }
      // (spilling: batch nstage-2's rows are copied out before batch
      // nstage, which may overwrite their temporary slots, is staged)
      if (nstage < nb && done >= nstage - 1 && (!spilling || nstore >= nstage - 1)) {
        if (ring_ok(a0, a1)) {
          stage(nstage, pa, a0, a1, ma);
          sync_set(kStaged, nstage + 1);
          ++nstage;
          ring_load(nstage * kBatch, a0, a1);
          pa = profit_at(nstage * kBatch + lane);
          ma = meta_at(nstage * kBatch + lane);
          progress = true;
        } else if (++spins > spin_limit) {
          ok = false;
          break;
        } else {
          ring_load(nstage * kBatch, a0, a1);
        }
      }
      if (progress) {
        idle = 0;
      } else {
        if (++idle > kLdsSpins) {
          ok = false;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    if (ok) return;
    sync_set(kStaged, -1);
    if (lane == 0)
      __hip_atomic_store(&d.cs[slot].status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return;
  }

  // ------------------------------------------------------- compute wave
  const int zero_off = slots * kStride;
#pragma unroll
  for (int c = 0; c < C; ++c) *(int64_t*)(lane_bytes + zero_off + c * kWave * 8) = 0;
  // x: the previous row D[i+1]; pre[u % 2]: the far skip row of step u,
  // read two steps ahead (padded steps 0 and 1 need none: step 0 is a leaf,
  // and a non-leaf step 1 skips to D[n+1], the zero row)
  int64_t x[C], pre[2][C];
  uint32_t acc[C];
#pragma unroll
  for (int c = 0; c < C; ++c) {
    x[c] = 0;
    pre[0][c] = 0;
    pre[1][c] = 0;
    acc[c] = 0;
  }
  // gather: lane u < kBatch reads the last cell (lane 63, cell C-1) of the
  // row step u was stored to
  constexpr int kLastCell = (C - 1) * kWave * 8 + (kWave - 1) * 8;
  barrier();
  // The compute wave issues ahead of other waves on its SIMD (another
  // block's I/O wave shares it at two blocks per compute unit).
  __builtin_amdgcn_s_setprio(2);

  // LDS address of this lane's cell 0 in row offset 0 (rows are addressed
  // as this plus a row's byte offset)
  const uint32_t lane_base =
      (uint32_t)(size_t)(__attribute__((address_space(3))) char*)lane_bytes;
  // t, sk of the previous step, whose choice bits are shifted into acc at
  // the start of the next step
  int64_t tp[C], skp[C];
  // Records of steps u..u+3 in flight, in a ring of kRq register sets that
  // runs across batches (kRq divides kBatch): a batch's record kBatch is
  // the next batch's record 0, and records 1 and 2 of the next batch are
  // read from its buffer after the staged count, a few steps ahead.
  constexpr int kRq = 4;
  static_assert(kBatch % kRq == 0, "record ring");
  pp_u32x4 rv[kRq];
  int staged_v;  // the staged count as loaded (made uniform where checked)
  auto view_of = [&](int buf) {
    return (const char*)(recs + buf * (kBatch + 1) * 2) + (lane == 0 ? sizeof(StepView) : 0);
  };
  auto rec_load = [&](int buf, int t) {
    rv[t % kRq] = *(const pp_u32x4*)(view_of(buf) + 2 * sizeof(StepView) * t);
  };
  staged_v = sync_load(kStaged);  // 1, or -1 if staging batch 0 failed
  rec_load(0, 0);
  rec_load(0, 1);
  rec_load(0, 2);

  // gather: lane u < kBatch reads the last cell of the row step u of a
  // batch was stored to, in groups of kProd steps.  At one cell per lane a
  // batch's values are handed to the I/O wave a few steps into the next
  // batch (or after the last one), when the last group's read has landed
  // without a wait; wider rows (eight groups to select from) hand off at
  // the end of the batch, which measures faster there.
  constexpr bool kDefer = C == 1;
  constexpr int kGroups = kBatch / kProd;
  int64_t gath_kept[kDefer ? kGroups : 1];  // carried into the next batch
#pragma unroll
  for (int q = 0; q < (kDefer ? kGroups : 1); ++q) gath_kept[q] = 0;
  // a batch's stage-ring values (lane u: step u's) to output buffer obuf
  // and the finished-batch count to `done`
  auto hand_off = [&](int64_t v, int obuf, int done) {
    if (kDefer || lane < kBatch) outv[obuf * kOutv + lane] = v;
    sync_set(kDone, done);
  };
  auto select_groups = [&](const int64_t (&g)[kDefer ? kGroups : 1]) {
    int64_t v = g[0];
#pragma unroll
    for (int q = 1; q < (kDefer ? kGroups : 1); ++q)
      if (lane >= q * kProd) v = g[q];
    return v;
  };
  constexpr int kHandOff = 2;  // step of the next batch that hands off
  static_assert(!kDefer || kHandOff + 1 < kProd, "hand-off before the next gather");

  // one batch; `buf` (b % 2, a compile-time constant) selects the record
  // and output buffers.  Returns false if the I/O wave gave up.
  auto batch = [&](auto bufc, int b) -> bool {
    constexpr int buf = decltype(bufc)::value;
    {
      int staged = __builtin_amdgcn_readfirstlane(staged_v);
      if (staged < b + 1) {
        // not staged when records 1 and 2 were read: wait, then read again
        uint32_t polls = 0;
        while (staged >= 0 && staged < b + 1) {
          if (++polls > kLdsSpins) {
            if (lane == 0)
              __hip_atomic_store(&d.cs[slot].status, 1, __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT);
            staged = -1;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
          staged = sync_get(kStaged);
        }
        if (staged < b + 1) return false;
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        rec_load(buf, 1);
        rec_load(buf, 2);
      }
    }
    const StepView* rec = recs + buf * (kBatch + 1) * 2;
    // gather addresses: lane u < kBatch, step u's rows word (at one cell
    // per lane read by every lane: lanes >= kBatch read words inside the
    // control area, and use 0)
    uint32_t gath_w = 0;
    if constexpr (kDefer) {
      const uint32_t gath_rw = rec[2 * lane].rows;
      gath_w = lane < kBatch ? gath_rw : 0u;
    } else {
      gath_w = lane < kBatch ? rec[2 * lane].rows : 0u;
    }
    const uint32_t gath_base = lane_base - lane * 8 + kLastCell;
    uint32_t gath_a = 0;
    // wider rows: each group's values are folded into gath_v one group
    // later (the read has landed by then), so no group array is kept
    int64_t gath_v = 0, gath_p = 0;
    auto step = [&](auto uc) {
      constexpr int u = decltype(uc)::value;
      if constexpr (u + 3 < kBatch) {
        rec_load(buf, u + 3);
      } else if constexpr (u + 3 == kBatch) {
        rec_load(buf, kBatch);  // = the next batch's record 0
      } else {
        // records 1, 2 of the next batch, after the staged count
        if constexpr (u + 3 == kBatch + 1) {
          staged_v = sync_load(kStaged);
          __atomic_signal_fence(__ATOMIC_SEQ_CST);
        }
        rec_load(1 - buf, u + 3 - kBatch);
      }
      const pp_u32x4 r = rv[u % kRq];
      const int64_t r0 = (int64_t)(((uint64_t)r.y << 32) | r.x);
      const uint64_t leaf = ((uint64_t)r.w << 32) | r.w;
      int64_t t[C], sk[C], y[C];
      // cell 0's take operand comes from the left lane (lane 0: r0 already
      // holds it); the previous step's choice bits go in first
      if constexpr (F64) {
        if constexpr (u > 0) acc[0] = shift_in_gt<true>(tp[0], skp[0], acc[0]);
        t[0] = take_f64(r0, x[C - 1]);
      } else if constexpr (u == 0) {
        t[0] = take_first_i64(r0, x[C - 1]);
      } else {
        t[0] = take_after_bit_i64(r0, x[C - 1], tp[0], skp[0], acc[0]);
      }
      // cells 1..C-1 add p itself, which lanes 1..63 hold; lane 0 (whose
      // view adds the boundary value) takes lane 1's by DPP wave_shl:1,
      // and lane 63, which has no right neighbour, keeps its own
      if constexpr (C > 1) {
        pp_int2 pq;
        pq.x = __builtin_amdgcn_update_dpp((int)r.x, (int)r.x, 0x130, 0xf, 0xf, false);
        pq.y = __builtin_amdgcn_update_dpp((int)r.y, (int)r.y, 0x130, 0xf, 0xf, false);
        const int64_t pl = join64(pq);
#pragma unroll
        for (int c = 1; c < C; ++c) {
          if constexpr (u > 0) acc[c] = shift_in_gt<F64>(tp[c], skp[c], acc[c]);
          t[c] = vadd<F64>(pl, x[c - 1]);
        }
      }
#pragma unroll
      for (int c = 0; c < C; ++c) {
        sk[c] = (int64_t)(((uint64_t)x[c] & leaf) | ((uint64_t)pre[u % 2][c] & ~leaf));
        if constexpr (FMAX)
          y[c] = max_nonneg_f64(sk[c], t[c]);
        else
          y[c] = t[c] > sk[c] ? t[c] : sk[c];
      }
      // the row goes to its slot if it is a later skip target, else to a
      // sink row
      {
        lds_i64* dst = lds_at(lds_row_lo(r.z, lane_base));
#pragma unroll
        for (int c = 0; c < C; ++c) dst[c * kWave] = y[c];
      }
      // skip row of step u+2 (high half of step u+1's rows word), read after
      // this store: it is row i-2's next(), produced at this step at the latest
      {
        const lds_i64* src = lds_at(lds_row_hi(rv[(u + 1) % kRq].z, lane_base));
#pragma unroll
        for (int c = 0; c < C; ++c) pre[u % 2][c] = src[c * kWave];
      }
      // the previous batch's ring values and count (batch 0: the count
      // stays 0 and buffer 1 gets values that batch 1 overwrites)
      if constexpr (kDefer && u == kHandOff) hand_off(select_groups(gath_kept), 1 - buf, b);
      if constexpr (u % kProd == kProd - 1) {
        constexpr int q = u / kProd;
        if constexpr (u == kProd - 1) gath_a = lds_row_lo(gath_w, gath_base);
        if constexpr (kDefer) {
          gath_kept[q] = *lds_at(gath_a);
        } else {
          if constexpr (q == 1) gath_v = gath_p;
          if constexpr (q > 1) gath_v = lane >= (q - 1) * kProd ? gath_p : gath_v;
          gath_p = *lds_at(gath_a);
        }
      }
#pragma unroll
      for (int c = 0; c < C; ++c) {
        tp[c] = t[c];
        skp[c] = sk[c];
        x[c] = y[c];
      }
    };
    unroll_steps(step, std::make_integer_sequence<int, kBatch>{});
    // choice bits of the batch's last step
#pragma unroll
    for (int c = 0; c < C; ++c) acc[c] = shift_in_gt<F64>(tp[c], skp[c], acc[c]);
    // the batch's choice words (and, unless deferred, its ring values)
#pragma unroll
    for (int c = 0; c < C; ++c) outb[(buf * C + c) * kWave + lane] = acc[c];
    if constexpr (!kDefer)
      hand_off(lane >= (kGroups - 1) * kProd ? gath_p : gath_v, buf, b + 1);
    return true;
  };
  bool ok = true;
  for (int b = 0; ok && b < nb; b += 2) {
    ok = batch(IC<0>{}, b);
    if (ok && b + 1 < nb) ok = batch(IC<1>{}, b + 1);
  }
  release_claim();
  if (!ok) {
    sync_set(kDone, -1);
    return;
  }
  if constexpr (kDefer) hand_off(select_groups(gath_kept), (nb - 1) % 2, nb);
  // D[1][k'] sits in stage (k'-1)/(64C), lane ((k'-1) mod 64C)/C, cell c.
  const int jj = kp - 1;
  if (jj / (kWave * C) == g) {
    const int rem = jj % (kWave * C);
    const int ln = rem / C, cc = rem % C;
    if (lane == ln) {
      int64_t v = 0;
#pragma unroll
      for (int c = 0; c < C; ++c)
        if (c == cc) v = x[c];
      d.cs[slot].dpval = v;
    }
  }
}

// ----------------------------------------------------------- backtrack --

// v_writelane_b32 (not exposed as a clang builtin): lane `lane` of the
// result is `val`, every other lane keeps `old`.
extern "C" __device__ int pp_writelane_i32(int val, int lane, int old) __asm(
    "llvm.amdgcn.writelane.i32");

// The backtrack walk through one staged super-window, in scalar code.
// Row sets of 32 consecutive rows (windows) are staged in LDS: for window k
// and lane l, the 16-byte table row of row q_lo + 32k + (l mod 32) at
// ace + 512k (chain mask, exit row at +4, the exit row's chain mask at +8),
// and the choice word of column l of the 64 columns the pass walks (a plane:
// a stage of one cell per lane, or a quarter or half of a wider one) at
// aw + 256k.  Exit rows past the last row are kCeEnd.  In window wk the walk
// reads those into registers, then finds the takes: the next take is the
// lowest set bit of (word of column rem & chain mask of q); it is recorded
// (bit of tm), the walk moves to the row after it and to column rem-1.
// Without a set bit the walk leaves the window at the chain's exit row.
// When the window changes, tm goes to lane wk of tw and is cleared.  The
// walk returns when rem wraps below zero (it leaves the plane) or when q
// leaves the super-window (wk >= 16; rows past the last one do).  On entry
// wk < 16, q lies in window wk, 0 <= rem < 64 and q < n.  Every pass raises
// q, so each window takes at most 32 passes.
//
// The walk keeps the two window sets in fixed registers
// (v48-v51: table rows of set P's window -- chain mask, exit row, the exit
// row's chain mask --, v56: its choice words; v52-v55 and v57: set N), so
// one 16-byte LDS read fetches a lane's table row.  A take is the lowest
// set bit of (mask of row r & word of column rem); both lookups of the next
// take are issued before the take's own bookkeeping.  A window is left
// either after a take at its last row (next window, row 0) or, with no
// take, at the exit row, whose chain mask comes with the row just left; in
// both cases the next window is usually the one already in the other set,
// and the walk continues there after one pair of lane reads.  Exit rows
// past the last row are kCeEnd, so they leave the super-window like any
// row beyond it.  Every pass raises the row, so the walk ends.
#define PP_W1_LOAD(CE, WD, IDX)                                  \
  "s_lshl_b32 %[off], %[" IDX "], 9\n\t"                         \
  "v_add_u32_e32 %[va], %[off], %[ace]\n\t"                      \
  "ds_read_b128 " CE ", %[va]\n\t"                               \
  "s_lshl_b32 %[off], %[" IDX "], 8\n\t"                         \
  "v_add_u32_e32 %[vb], %[off], %[aw]\n\t"                       \
  "ds_read_b32 " WD ", %[vb]\n\t"
// window wk + 1 (or 15 past the last one, never walked) into a set
#define PP_W1_NEXT(CE, WD)                                       \
  "s_add_u32 %[nx], %[wk], 1\n\t"                                \
  "s_min_u32 %[nx], %[nx], 15\n\t"                               \
  PP_W1_LOAD(CE, WD, "nx")
// Takes inside the window of set S (labels T1-T4); O is the other set.
// On entry m = chain mask of row r, w = word of column rem, and nx =
// min(wk + 1, 15), the window the other set holds (an exit row in window 16
// therefore leaves the super-window).
#define PP_W1_SET(T, CE, CM, CX, CXM, WS, OCM, OWS, OT, DIR)     \
  T "1:\n\t"                                                     \
  "s_and_b32 %[t], %[m], %[w]\n\t"                               \
  "s_cbranch_scc0 " T "3f\n\t"                                   \
  "s_ff1_i32_b32 %[t], %[t]\n\t"                                 \
  "s_add_u32 %[r], %[t], 1\n\t"                                  \
  "s_bitset1_b32 %[tm], %[t]\n\t"                                \
  "s_sub_u32 %[rem], %[rem], 1\n\t"                              \
  "v_readlane_b32 %[m], " CM ", %[r]\n\t"                        \
  "v_readlane_b32 %[w], " WS ", %[rem]\n\t"                      \
  "s_cbranch_scc1 " T "4f\n\t"                                   \
  "s_cmp_lg_u32 %[r], 32\n\t"                                    \
  "s_cbranch_scc1 " T "1b\n\t"                                   \
  /* a take at the last row: the next window, row 0 */           \
  "s_mov_b32 m0, %[wk]\n\t"                                      \
  "v_writelane_b32 %[tw], %[tm], m0\n\t"                         \
  "s_mov_b32 %[tm], 0\n\t"                                       \
  "s_add_u32 %[wk], %[wk], 1\n\t"                                \
  "s_add_u32 %[wlo], %[wlo], 32\n\t"                             \
  "s_cmp_ge_u32 %[wk], 16\n\t"                                   \
  "s_cbranch_scc1 97f\n\t"                                       \
  "s_mov_b32 %[r], 0\n\t"                                        \
  "s_waitcnt lgkmcnt(0)\n\t"                                     \
  "v_readlane_b32 %[m], " OCM ", 0\n\t"                          \
  "v_readlane_b32 %[w], " OWS ", %[rem]\n\t"                     \
  PP_W1_NEXT(CE, WS)                                             \
  "s_branch " OT "1" DIR "\n\t"                                  \
  /* no take: the exit row and its chain mask */                 \
  /* (the other set's word of column rem is read before it is */ \
  /* known to be the window: unused otherwise) */                 \
  T "3:\n\t"                                                     \
  "s_waitcnt lgkmcnt(0)\n\t"                                     \
  "v_readlane_b32 %[q], " CX ", %[r]\n\t"                        \
  "v_readlane_b32 %[m], " CXM ", %[r]\n\t"                       \
  "v_readlane_b32 %[w], " OWS ", %[rem]\n\t"                     \
  "s_mov_b32 m0, %[wk]\n\t"                                      \
  "v_writelane_b32 %[tw], %[tm], m0\n\t"                         \
  "s_mov_b32 %[tm], 0\n\t"                                       \
  "s_sub_u32 %[wk], %[q], %[qlo]\n\t"                            \
  "s_lshr_b32 %[wk], %[wk], 5\n\t"                               \
  /* nx = min(wk + 1, 15) of the window left: the other set's */  \
  "s_cmp_lg_u32 %[wk], %[nx]\n\t"                                \
  "s_cbranch_scc1 15f\n\t"                                       \
  "s_add_u32 %[wlo], %[wlo], 32\n\t"                             \
  "s_sub_u32 %[r], %[q], %[wlo]\n\t"                             \
  PP_W1_NEXT(CE, WS)                                             \
  "s_branch " OT "1" DIR "\n\t"                                  \
  /* the take used the stage's first column: leave the stage */  \
  T "4:\n\t"                                                     \
  "s_add_u32 %[q], %[wlo], %[r]\n\t"                             \
  "s_cmp_lg_u32 %[r], 32\n\t"                                    \
  "s_cbranch_scc1 99f\n\t"                                       \
  "s_mov_b32 m0, %[wk]\n\t"                                      \
  "v_writelane_b32 %[tw], %[tm], m0\n\t"                         \
  "s_mov_b32 %[tm], 0\n\t"                                       \
  "s_add_u32 %[wk], %[wk], 1\n\t"                                \
  "s_branch 99f\n\t"

__device__ __forceinline__ void walk_sw_c1(uint32_t& q, uint32_t& rem, uint32_t& tm,
                                           uint32_t& wk, uint32_t& tw, uint32_t qlo,
                                           uint32_t ace, uint32_t aw) {
  uint32_t r, m, w, t, off, wlo, nx, sm0, va, vb;
  asm volatile(
      "s_mov_b32 %[sm0], m0\n\t"
      // (re)load: window wk into set P, wk + 1 into set N; row r of wk
      "10:\n\t"
      "s_waitcnt lgkmcnt(0)\n\t"
      PP_W1_LOAD("v[48:51]", "v56", "wk")
      "s_add_u32 %[nx], %[wk], 1\n\t"
      "s_min_u32 %[nx], %[nx], 15\n\t"
      PP_W1_LOAD("v[52:55]", "v57", "nx")
      "s_lshl_b32 %[wlo], %[wk], 5\n\t"
      "s_add_u32 %[wlo], %[wlo], %[qlo]\n\t"
      "s_sub_u32 %[r], %[q], %[wlo]\n\t"
      "s_waitcnt lgkmcnt(2)\n\t"
      "v_readlane_b32 %[m], v48, %[r]\n\t"
      "v_readlane_b32 %[w], v56, %[rem]\n\t"
      "s_branch 11f\n\t"
      PP_W1_SET("1", "v[48:51]", "v48", "v49", "v50", "v56", "v52", "v57", "2", "f")
      PP_W1_SET("2", "v[52:55]", "v52", "v53", "v54", "v57", "v48", "v56", "1", "b")
      // the exit row is not in the next window: leave the super-window, or
      // reload both sets around it
      "15:\n\t"
      "s_cmp_ge_u32 %[wk], 16\n\t"
      "s_cbranch_scc1 99f\n\t"
      "s_branch 10b\n\t"
      // a take at the super-window's last row
      "97:\n\t"
      "s_mov_b32 %[q], %[wlo]\n\t"
      // no LDS read may still be landing in a register the compiler reuses
      "99:\n\t"
      "s_waitcnt lgkmcnt(0)\n\t"
      "s_mov_b32 m0, %[sm0]"
      : [q] "+s"(q), [rem] "+s"(rem), [tm] "+s"(tm), [wk] "+s"(wk), [tw] "+v"(tw),
        [r] "=&s"(r), [m] "=&s"(m), [w] "=&s"(w), [t] "=&s"(t), [off] "=&s"(off),
        [wlo] "=&s"(wlo), [nx] "=&s"(nx), [sm0] "=&s"(sm0), [va] "=&v"(va), [vb] "=&v"(vb)
      : [qlo] "s"(qlo), [ace] "v"(ace), [aw] "v"(aw)
      : "scc", "memory", "v48", "v49", "v50", "v51", "v52", "v53", "v54", "v55", "v56",
        "v57");
}
#undef PP_W1_SET
#undef PP_W1_NEXT
#undef PP_W1_LOAD


// Acceptance (greedy: always; refinement: DP value > incumbent value, which
// by Proposition 1 is G(T_-h, T'_h) > G(T)) and, when accepted, the walk
// from (i=1, j=k'): take b_i if its choice bit is set (i+1, j-1), else jump
// to next(i).
//
// A choice word of one sweep batch holds 32 consecutive rows -- a window,
// row q at bit q mod 32 (the padded step count is a multiple of 32) -- of
// one cell column.  While j stays fixed the walk visits q, next(q),
// next(next(q)), ...; the rows of that sequence inside q's window are one
// precomputed mask, so the next take is the lowest set bit of (column word
// & mask), and without one the walk leaves the window at the sequence's
// precomputed exit row: the scalar walk advances per take, not per row.
// Rows are staged in super-windows of 512: the words of the current stage
// and the masks and exit rows of the 512 rows go to LDS.  While one is
// walked, two successors are loaded from memory into registers: the next
// super-window of the same stage (rows only increase along the walk) and
// the same super-window of the stage below (j only decreases, and leaves
// the stage after at most 64C takes).  Taken rows are
// gathered per window (lane k of tw: window k of the super-window) and
// written as a bitmap when the walk leaves the super-window.
template <int C>
__global__ void __launch_bounds__(64) k_backtrack(ChainSet set, DevState d,
                                                  int mode) {
  constexpr int kWin = kDpBatch;        // rows per choice word
  constexpr int kSwWin = 16;            // windows per super-window
  constexpr int kSw = kWin * kSwWin;    // rows per super-window
  static_assert(kSw == kCeBlock, "the chain table is padded per super-window");
  constexpr int kW = C * 4;             // 16-byte word loads per lane
  static_assert(kWin == 32 && kSwWin == 16, "the scalar walk's window layout");
  // choice words by plane (64 consecutive columns of the stage), window and
  // column within the plane
  __shared__ __attribute__((aligned(16))) uint32_t s_words[C][kSwWin][kWave];
  // chain mask, exit row, the exit row's chain mask, 0
  __shared__ __attribute__((aligned(16))) uint32_t s_ce[kSw][4];
  const int ci = blockIdx.x;
  const int lane = threadIdx.x;
  const int64_t slot = set.slot[ci];
  const int kp = set.kprime[ci];
  const int n = d.n;
  ChainState* st = d.cs + slot;
  if (st->skip) {
    if (lane == 0) {
      st->accept = 0;
      st->inc = 0;
    }
    return;
  }
  if (lane == 0) {  // worker h's DP ran: its inputs are current again
    const int h = set.worker[ci];
    st->dirty[h >> 5] &= ~(1u << (h & 31));
  }
  const int64_t dpval = st->dpval;
  bool accept;
  if (d.f64) {
    // Real-valued costs: the decision, on the exact G of the placement with
    // T'_h against the exact G(T) + eps (Algorithm 1's test evaluated from
    // scratch), is k_gexact_final's, which also sets the acceptance marks.
    // A refinement update is rejected here, without its walk, when its DP
    // value stays below the incumbent's value + eps by more than E, a bound
    // on how far the rounded sums can be from that exact difference of G
    // (Proposition 1): each marginal is within (M + 4) u W_b of the exact
    // difference of its chunk's rounded terms (u = 2^-53, W_b = sum over
    // requesters of Lambda * w), each of the two sums of at most k' of them
    // adds k' u of its total, and denormal terms add at most 2^-1074 per
    // rounding.
    const double dv = as_f(dpval), inc = as_f(st->inc), wsum = as_f(st->wsum);
    bool early = false;
    if (mode == kModeRefine) {
      const double u = 0x1p-53;
      const double e = 1.25 * (d.m + 8.0 + 2.0 * kp) * u * wsum + 2.0 * u * d.eps +
                       (double)n * (d.m + 4.0) * 0x1p-1070;
      early = dv + e < inc + d.eps;
    }
    if (lane == 0) {
      st->accept = 0;
      st->inc = 0;
      st->wsum = 0;
      st->rejected = early ? 1 : 0;
    }
    if (early) return;
    const int nwords = d.npad / 32;
    uint32_t* selw = d.sel + slot * nwords;
    for (int q = lane; q < nwords; q += kWave) selw[q] = 0;
    if (kp <= 0) return;
    accept = true;
  } else {
    const int64_t inc = st->inc;
    accept = (mode == kModeGreedy) || (dpval > inc);
    if (lane == 0) {
      st->accept = accept ? 1 : 0;
      st->inc = 0;
      if (mode == kModeRefine && accept) st->accepts += 1;
    }
  }
  if (!accept) return;
  const int nwords = d.npad / 32;
  uint32_t* selw = d.sel + slot * nwords;
  if (!d.f64) {
    if (lane == 0) {
      // every other worker's marginals change with worker h's set
      const int h = set.worker[ci];
#pragma unroll
      for (int q = 0; q < 8; ++q) st->dirty[q] |= q == (h >> 5) ? ~(1u << (h & 31)) : ~0u;
    }
    for (int q = lane; q < nwords; q += kWave) selw[q] = 0;
    if (kp <= 0) return;
  }

  const int nwin = (n + kWin - 1) / kWin;  // windows = sweep batches
  const int64_t cstride = 2 * (int64_t)d.npad;
  const uint32_t* bw = (const uint32_t*)d.bits + slot * d.stages * (int64_t)C * cstride;

  // Window k of super-window sw is sweep batch nwin-1-(16 sw + k), so the
  // 16 windows are 16 consecutive batches: 64 lanes x 4 KB per cell, read
  // as four 16-byte loads per lane (load i, lane l: batch blo + 4i + l/16 =
  // window 15 - 4i - l/16, columns 4(l mod 16) .. +3).  Windows past the
  // last row are never walked; their loads are clamped into range.
  auto load_words = [&](int sw, int g, pp_u32x4 (&w)[kW]) {
    const int blo = nwin - kSwWin - sw * kSwWin;
    const uint32_t* base = bw + (int64_t)g * C * cstride + 4 * (lane % 16);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int b = max(blo + 4 * i + lane / 16, 0);
#pragma unroll
      for (int c = 0; c < C; ++c)
        w[c * 4 + i] = *(const pp_u32x4*)(base + c * cstride + (int64_t)b * kWave);
    }
  };
  // table rows of the super-window's 512 rows, one 16-byte row per load
  // (the host pads the table with empty rows through one super-window past
  // the end)
  auto load_chain = [&](int sw, pp_u32x4 (&ce)[8]) {
    const pp_u32x4* src = (const pp_u32x4*)d.ce + (int64_t)sw * kSw;
#pragma unroll
    for (int i = 0; i < 8; ++i) ce[i] = src[i * kWave + lane];
  };
  // (a load holds sweep lanes 4(l mod 16) .. +3 of one cell c; sweep lane
  // u's cell c is column uC + c of the stage)
  auto words_to_lds = [&](const pp_u32x4 (&w)[kW]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = kSwWin - 1 - (4 * i + lane / 16);
      if constexpr (C == 1) {
        *(pp_u32x4*)&s_words[0][k][4 * (lane % 16)] = w[i];
      } else {
#pragma unroll
        for (int c = 0; c < C; ++c)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int col = (4 * (lane % 16) + e) * C + c;
            s_words[col / kWave][k][col % kWave] = w[c * 4 + i][e];
          }
      }
    }
  };
  auto chain_to_lds = [&](const pp_u32x4 (&ce)[8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i) ((pp_u32x4*)&s_ce[0][0])[i * kWave + lane] = ce[i];
  };
  // LDS addresses the walk reads from: lane l's row (l mod 32) of window 0
  // and the word of column l of window 0 in plane 0 (plane p: + p * kPlane)
  const uint32_t ace = (uint32_t)(size_t)(__attribute__((address_space(3))) uint32_t*)&s_ce[lane % kWin][0];
  const uint32_t aw = (uint32_t)(size_t)(__attribute__((address_space(3))) uint32_t*)&s_words[0][0][lane];
  constexpr uint32_t kPlane = kSwWin * kWave * sizeof(uint32_t);
  // this super-window's take masks to the bitmap
  auto store_takes = [&](int sw, uint32_t tw) {
    const int idx = sw * kSwWin + lane;
    if (lane < kSwWin && idx < nwords) selw[idx] = tw;
  };

  int q = 0, j = kp;
  int pl = (j - 1) / kWave;  // plane of column j (64 columns each)
  int g = pl / C;            // its stage
  int sw = 0;
  pp_u32x4 wb[kW];  // next super-window, same stage
  pp_u32x4 wd[kW];  // same super-window, stage below
  pp_u32x4 cb[8];
  load_words(0, g, wb);
  load_chain(0, cb);
  words_to_lds(wb);
  chain_to_lds(cb);
  __syncthreads();
  static_assert(C == 1 || C == 2 || C == 4, "one, two or four cells per lane");
  uint32_t tw = 0, tm = 0;
  for (;;) {
    // both successors, in flight while this super-window is walked
    load_words(sw + 1, g, wb);
    if (g > 0) load_words(sw, g - 1, wd);
    load_chain(sw + 1, cb);
    int sw_n = sw, pl_n = pl;
    bool done = false;
    for (;;) {  // the planes of stage g walked inside super-window sw
      const int jlo = pl * kWave + 1;
      uint32_t uq = (uint32_t)q, urem = (uint32_t)(j - jlo);
      uint32_t wk = (uint32_t)(q - sw * kSw) / kWin;
      walk_sw_c1(uq, urem, tm, wk, tw, (uint32_t)(sw * kSw), ace,
                 aw + (uint32_t)(pl % C) * kPlane);
      q = (int)uq;
      j = jlo + (int)urem;
      if (q >= n || j == 0) {
        if (wk < (uint32_t)kSwWin) tw = (uint32_t)pp_writelane_i32((int)tm, (int)wk, (int)tw);
        store_takes(sw, tw);
        done = true;
        break;
      }
      // the walk left the plane or the super-window
      sw_n = q / kSw;
      pl_n = (j - 1) / kWave;
      if (C == 1 || sw_n != sw || pl_n / C != g) break;
      pl = pl_n;  // the next plane of the stage: its words are staged already
    }
    if (done) break;
    const int g_n = pl_n / C;
    if (sw_n != sw) {
      store_takes(sw, tw);  // the last window's takes are in tw already
      tw = 0;
    }
    bool below = false;
    if (g_n == g && sw_n == sw + 1) {
      // the prefetched super-window
    } else if (g_n == g) {
      load_words(sw_n, g_n, wb);
      load_chain(sw_n, cb);
    } else if (sw_n == sw) {
      below = true;  // the prefetched stage below
    } else {
      load_words(sw_n, g_n, wb);
      load_chain(sw_n, cb);
    }
    __syncthreads();
    if (below)
      words_to_lds(wd);
    else
      words_to_lds(wb);
    if (sw_n != sw) chain_to_lds(cb);
    __syncthreads();
    sw = sw_n;
    g = g_n;
    pl = pl_n;
  }
}

// -------------------------------------------------------------- commit --

// Adopt T'_h where accepted: write the new membership and refresh the top-2
// holder state of every chunk whose membership changed.  A block holds
// kCommitThreads / M chunks times M requesters (requester-major, so each
// requester's loads are contiguous); each thread updates one requester's
// top-2, and the new membership is written after a barrier.  Only worker
// h's membership changes, so the new state follows from the old one and
// h's saving q_h: when h joins, q_h is inserted (top-2 values of the
// multiset, lowest holder id among the maxima); when h leaves and was
// neither the best holder nor tied with the second value (q_h < v2), the
// state is unchanged.  Otherwise (h leaves as h1, or with q_h == v2) the
// thread rebuilds the top-2 over all holders, O(M).
constexpr int kCommitThreads = 256;

__global__ void __launch_bounds__(kCommitThreads) k_commit(ChainSet set, DevState d,
                                                            int mode) {
  const int ci = blockIdx.y;
  const int64_t s = set.slot[ci];
  if (!d.cs[s].accept) return;
  const int h = set.worker[ci];
  const int m = d.m;
  const int64_t n = d.n;
  const int cpb = kCommitThreads / m;  // chunks per block (m <= 255)
  const int r = threadIdx.x / cpb;
  const int64_t i = (int64_t)blockIdx.x * cpb + threadIdx.x % cpb;
  const int64_t mn = (int64_t)m * n;
  const uint8_t* t = d.tgt + s * mn;
  uint8_t* th = d.tgt + s * mn + (int64_t)h * n;
  bool changed = false;
  uint8_t nv = 0;
  if (r < m && i < n) {
    nv = (uint8_t)((d.sel[s * (d.npad / 32) + i / 32] >> (i % 32)) & 1u);
    changed = nv != th[i];
  }
  if (!__syncthreads_or(changed)) return;
  if (changed) {
    const int64_t o = s * mn + (int64_t)r * n + i;
    const int64_t wr = d.w[(int64_t)r * n + i];
    auto q_of = [&](int l) -> int64_t {
      if (l == r) return wr;
      const int64_t fv = d.f[((int64_t)l * m + r) * n + i];
      return d.f64 ? as_i(dpos(as_f(wr) - as_f(fv))) : imax(wr - fv, 0);
    };
    const int64_t qh = q_of(h);
    int64_t b1 = d.v1[o], b2 = d.v2[o];
    int hb = d.h1[o];
    // savings are non-negative (doubles: finite, +0 for none), so their
    // bit patterns compare like the values
    bool rebuild = false;
    if (nv) {
      if (hb == kNoHolder) {
        b1 = qh;
        b2 = 0;
        hb = h;
      } else if (qh > b1) {
        b2 = b1;
        b1 = qh;
        hb = h;
      } else if (qh == b1) {
        b2 = b1;
        hb = h < hb ? h : hb;
      } else if (qh > b2) {
        b2 = qh;
      }
    } else {
      rebuild = hb == h || qh >= b2;
    }
    if (rebuild) {
      b1 = 0;
      b2 = 0;
      hb = kNoHolder;
#pragma unroll 8
      for (int l = 0; l < m; ++l) {
        if (l == h || t[(int64_t)l * n + i] == 0) continue;
        const int64_t q = q_of(l);
        if (hb == kNoHolder || q > b1) {
          b2 = (hb == kNoHolder) ? b2 : b1;
          b1 = q;
          hb = l;
        } else if (q > b2) {
          b2 = q;
        }
      }
    }
    d.v1[o] = b1;
    d.v2[o] = b2;
    d.h1[o] = (uint8_t)hb;
  }
  __syncthreads();  // every requester has read the old membership row
  if (changed && r == 0) th[i] = nv;
}

// Speculative refinement, after the decisions (one block per start): the
// workers in `ran` swept against the start's unchanged placement (their
// inputs are current); if a later position was accepted in spare slot
// `from`, slot s takes its selection and acceptance as k_backtrack leaves
// them for an update run in slot s itself, so that k_commit can adopt it
// there.
__global__ void __launch_bounds__(256) k_adopt(AdoptSet set, DevState d) {
  const int ci = blockIdx.x;
  const int32_t s = set.slot[ci], from = set.from[ci], h = set.worker[ci];
  ChainState* st = d.cs + s;
  if (from >= 0) {
    const int nwords = d.npad / 32;
    const uint32_t* src = d.sel + (int64_t)from * nwords;
    uint32_t* dst = d.sel + (int64_t)s * nwords;
    for (int q = threadIdx.x; q < nwords; q += blockDim.x) dst[q] = src[q];
    if (d.f64) {
      // the exact G with the adopted replacement becomes the start's G
      for (int q = threadIdx.x; q < kExLimbs; q += blockDim.x)
        d.gx[(s * 2) * kExLimbs + q] = d.gx[((int64_t)from * 2 + 1) * kExLimbs + q];
    }
  }
  if (threadIdx.x == 0) {
#pragma unroll
    for (int q = 0; q < 8; ++q) st->dirty[q] &= ~set.ran[ci][q];
    if (from >= 0) {
      const ChainState& fs = d.cs[from];
      st->accept = 1;
      st->inc = 0;
      st->dpval = fs.dpval;
      st->accepts += 1;
#pragma unroll
      for (int q = 0; q < 8; ++q)
        st->dirty[q] |= q == (h >> 5) ? ~(1u << (h & 31)) : ~0u;
      st->dirty[h >> 5] &= ~(1u << (h & 31));
    }
  }
}

// The first greedy update of a start (position 0, every worker's set
// empty) is the standalone solve of its worker (same profits, same DP), so
// it adopts that solve's selection, saved in `sel0` (row h: worker h),
// instead of sweeping again; the marks are those the walk would set (the
// real-valued decision and its marks follow in k_gexact_final).
__global__ void __launch_bounds__(256) k_take_standalone(ChainSet set, DevState d,
                                                         const uint32_t* __restrict__ sel0) {
  const int ci = blockIdx.x;
  const int64_t s = set.slot[ci];
  const int h = set.worker[ci];
  const int nwords = d.npad / 32;
  const uint32_t* src = sel0 + (int64_t)h * nwords;
  uint32_t* dst = d.sel + s * nwords;
  for (int q = threadIdx.x; q < nwords; q += blockDim.x) dst[q] = src[q];
  if (threadIdx.x == 0) {
    ChainState* st = d.cs + s;
    st->dirty[h >> 5] &= ~(1u << (h & 31));
    st->inc = 0;
    if (d.f64) {
      st->accept = 0;
      st->wsum = 0;
      st->rejected = 0;
    } else {
      st->accept = 1;
#pragma unroll
      for (int q = 0; q < 8; ++q) st->dirty[q] |= q == (h >> 5) ? ~(1u << (h & 31)) : ~0u;
    }
  }
}

// Row h of slot `dst`'s placement := the backtracked selection of chain
// (slot, h), for every chain of the set (the per-worker comparator
// candidates are solved in scratch slots and assembled here).
__global__ void k_assemble(ChainSet set, DevState d, int64_t dst) {
  const int ci = blockIdx.y;
  const int64_t s = set.slot[ci];
  const int h = set.worker[ci];
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i >= d.n) return;
  d.tgt[(dst * d.m + h) * (int64_t)d.n + i] =
      (uint8_t)((d.sel[s * (d.npad / 32) + i / 32] >> (i % 32)) & 1u);
}

// Requester-side inputs (Sec. III-B): f[src][dst][b] is the same for every
// src != dst.  Sets *mismatch when some entry differs.
__global__ void k_requester_check(const int64_t* __restrict__ f, int32_t n,
                                  int32_t m, int32_t* mismatch) {
  const int64_t mn = (int64_t)m * n;
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < mn;
       x += (int64_t)gridDim.x * blockDim.x) {
    const int dst = (int)(x / n);
    const int64_t b = x % n;
    const int first = dst == 0 ? 1 : 0;
    const int64_t ref = f[((int64_t)first * m + dst) * n + b];
    bool diff = false;
    for (int src = first + 1; src < m; ++src)
      if (src != dst && f[((int64_t)src * m + dst) * n + b] != ref) diff = true;
    if (diff) *mismatch = 1;
  }
}

// One-time cost of the chunks slot `prop` places that slot `inc` does not
// hold at the same worker (the re-planning rule of Sec. IV-D): each pays the
// cheaper of recomputation and a fetch from a worker holding it in `inc`.
// Exact per-block sums (128-bit) go to partial[blockIdx.x].
__global__ void __launch_bounds__(256) k_mat_cost(DevState d, int64_t inc, int64_t prop,
                                                  unsigned __int128* partial) {
  const int64_t n = d.n, mn = (int64_t)d.m * n;
  const uint8_t* ti = d.tgt + inc * mn;
  const uint8_t* tp = d.tgt + prop * mn;
  if (d.f64) {
    // the same minimum on bit patterns (non-negative doubles order like
    // them); the cost summed exactly, lazy per-block partials of kExLimbs
    // 64-bit limbs
    __shared__ unsigned long long acc[kExLimbs];
    for (int q = threadIdx.x; q < kExLimbs; q += blockDim.x) acc[q] = 0;
    __syncthreads();
    ExWindow win;
    for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < mn;
         x += (int64_t)gridDim.x * blockDim.x) {
      if (!tp[x] || ti[x]) continue;
      const int r = (int)(x / n);
      const int64_t i = x % n;
      int64_t c = d.w[x];
      for (int h = 0; h < d.m; ++h)
        if (h != r && ti[(int64_t)h * n + i]) {
          const int64_t fh = d.f[((int64_t)h * d.m + r) * n + i];
          if (fh < c) c = fh;
        }
      ex_accumulate(acc, win, as_f(c));
    }
    ex_flush(acc, win);
    __syncthreads();
    uint64_t* out = (uint64_t*)partial + (int64_t)blockIdx.x * kExLimbs;
    for (int q = threadIdx.x; q < kExLimbs; q += blockDim.x) out[q] = acc[q];
    return;
  }
  unsigned __int128 acc = 0;
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < mn;
       x += (int64_t)gridDim.x * blockDim.x) {
    if (!tp[x] || ti[x]) continue;
    const int r = (int)(x / n);
    const int64_t i = x % n;
    int64_t c = d.w[x];
    for (int h = 0; h < d.m; ++h)
      if (h != r && ti[(int64_t)h * n + i]) {
        const int64_t fh = d.f[((int64_t)h * d.m + r) * n + i];
        if (fh < c) c = fh;
      }
    acc += (uint64_t)c;
  }
  __shared__ unsigned __int128 part[256];
  part[threadIdx.x] = acc;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) part[threadIdx.x] += part[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) partial[blockIdx.x] = part[0];
}

// ----------------------------------------------------------- objective --

// F_pair(T) = sum_{m,b} Lambda_m(b) * v1_m(b)   (Eq. 6), integer costs.
__global__ void __launch_bounds__(256) k_objective(ChainSet set, DevState d) {
  const int ci = blockIdx.y;
  const int64_t s = set.slot[ci];
  const int64_t mn = (int64_t)d.m * d.n;
  int64_t acc = 0;
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < mn;
       x += (int64_t)gridDim.x * blockDim.x)
    acc += d.lam[x] * d.v1[s * mn + x];
  const int64_t t = block_sum(acc);
  if (threadIdx.x == 0 && t)
    atomicAdd((unsigned long long*)&d.cs[s].obj, (unsigned long long)t);
}

// Real-valued costs: G (Eq. 6) as the exact sum of its rounded terms, so
// that every comparison of objectives is independent of summation order.
// replace = 0: the slot's own placement, terms Lambda_r(b) * v1_r(b).
// replace = 1: the update's placement, worker h's set replaced by the
// backtracked selection T'_h: terms Lambda_r(b) * max(v_r^{(-h)}(b),
// [b in T'_h] q_{r<-h}(b)), v^{(-h)} from the source slot's top-2 holder
// state (the same values the oracle's maximum over holders gives).
// Per-block lazy partial sums go to d.gxp.
__global__ void __launch_bounds__(256) k_gexact(ChainSet set, DevState d, int replace) {
  const int ci = blockIdx.y;
  const int64_t s = set.slot[ci];
  if (replace && (d.cs[s].skip || d.cs[s].rejected)) return;  // already rejected
  __shared__ unsigned long long acc[kExLimbs];
  for (int q = threadIdx.x; q < kExLimbs; q += blockDim.x) acc[q] = 0;
  __syncthreads();
  const int64_t ps = set.src[ci];
  const int h = set.worker[ci];
  const int64_t n = d.n, mn = (int64_t)d.m * n;
  const uint32_t* selw = d.sel + s * (d.npad / 32);
  ExWindow win;
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < mn;
       x += (int64_t)gridDim.x * blockDim.x) {
    double best;
    if (replace) {
      const int r = (int)(x / n);
      const int64_t i = x - (int64_t)r * n;
      const int64_t o = ps * mn + x;
      best = as_f((d.h1[o] == h) ? d.v2[o] : d.v1[o]);
      if ((selw[i >> 5] >> (i & 31)) & 1u) {
        const double q = as_f(saving(d, h, r, i));
        best = q > best ? q : best;
      }
    } else {
      best = as_f(d.v1[s * mn + x]);
    }
    ex_accumulate(acc, win, as_f(d.lam[x]) * best);
  }
  ex_flush(acc, win);
  __syncthreads();
  if (threadIdx.x == 0) {  // carry the block's limbs: each below 2^32 after
    unsigned long long carry = 0;
    for (int q = 0; q < kExLimbs; ++q) {
      const unsigned long long v = acc[q] + carry;
      acc[q] = v & 0xFFFFFFFFull;
      carry = v >> 32;
    }
  }
  __syncthreads();
  uint64_t* part = d.gxp + ((int64_t)ci * d.gx_blocks + blockIdx.x) * kExLimbs;
  for (int q = threadIdx.x; q < kExLimbs; q += blockDim.x) part[q] = acc[q];
}

// One block per chain: the exact G from k_gexact's partials (carried into
// canonical limbs), then
//   kModeGreedy: the update is adopted: gx[slot][0] = G, acceptance marks;
//   kModeRefine: Algorithm 1's test, exact G(T_-h, T'_h) > exact G(T) +
//                eps with G(T) that of the source slot; on acceptance the
//                replacement is counted, the other workers' inputs marked
//                stale, and (in the start's own slot) G(T) updated;
//   otherwise:   the slot's objective, gx[slot][0] = G and its nearest
//                double in cs.obj.
// gx[slot][1] always receives G.
__global__ void __launch_bounds__(256) k_gexact_final(ChainSet set, DevState d, int mode,
                                                      int nblocks) {
  const int ci = blockIdx.x;
  const int64_t s = set.slot[ci];
  const bool update = mode == kModeGreedy || mode == kModeRefine;
  if (update && (d.cs[s].skip || d.cs[s].rejected)) return;
  // the blocks' partials are carried limbs (each below 2^32), so a limb's
  // sum over at most kGexactBlocks of them stays below 2^41
  __shared__ unsigned long long tot[kExLimbs];
  __shared__ uint32_t g[kExLimbs];
  for (int q = threadIdx.x; q < kExLimbs; q += blockDim.x) tot[q] = 0;
  __syncthreads();
  const uint64_t* part = d.gxp + (int64_t)ci * d.gx_blocks * kExLimbs;
  const int count = nblocks * kExLimbs;
  constexpr int kUnroll = 4;  // loads in flight per thread
  for (int x0 = threadIdx.x; x0 < count; x0 += kUnroll * blockDim.x) {
    uint64_t v[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      const int x = x0 + k * blockDim.x;
      v[k] = x < count ? part[x] : 0;
    }
#pragma unroll
    for (int k = 0; k < kUnroll; ++k)
      if (v[k]) atomicAdd(&tot[(x0 + k * blockDim.x) % kExLimbs], (unsigned long long)v[k]);
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  unsigned long long carry = 0;
  for (int q = 0; q < kExLimbs; ++q) {
    const unsigned long long v = tot[q] + carry;
    g[q] = (uint32_t)v;
    carry = v >> 32;
  }
  uint32_t* cur = d.gx + (s * 2) * kExLimbs;
  uint32_t* nxt = d.gx + (s * 2 + 1) * kExLimbs;
  for (int q = 0; q < kExLimbs; ++q) nxt[q] = g[q];
  ChainState* st = d.cs + s;
  if (!update) {
    for (int q = 0; q < kExLimbs; ++q) cur[q] = g[q];
    st->obj = (int64_t)ex_round_bits(g);
    return;
  }
  const int64_t ps = set.src[ci];
  bool accept = true;
  if (mode == kModeRefine) {
    uint32_t bar[kExLimbs];
    const uint32_t* gs = d.gx + (ps * 2) * kExLimbs;
    for (int q = 0; q < kExLimbs; ++q) bar[q] = gs[q];
    ex_add_double(bar, d.eps);
    accept = ex_cmp(g, bar) > 0;
  }
  st->accept = accept ? 1 : 0;
  if (!accept) return;
  if (mode == kModeRefine) st->accepts += 1;
  const int h = set.worker[ci];
  for (int q = 0; q < 8; ++q) st->dirty[q] |= q == (h >> 5) ? ~(1u << (h & 31)) : ~0u;
  if (s == ps)
    for (int q = 0; q < kExLimbs; ++q) cur[q] = g[q];
}

inline dim3 grid1(int64_t work, int bs, int rows) {
  int64_t b = (work + bs - 1) / bs;
  if (b < 1) b = 1;
  return dim3((unsigned)b, (unsigned)rows);
}

}  // namespace

// ---------------------------------------------------------- launchers ---

hipError_t launch_gather(const int64_t* src, int64_t* dst, int32_t rows,
                         int32_t n, const int32_t* order, hipStream_t st) {
  hipLaunchKernelGGL(k_gather, grid1(n, 256, rows), dim3(256), 0, st, src, dst,
                     n, order);
  return hipGetLastError();
}

hipError_t launch_gather_inputs(const int64_t* lam, const int64_t* w, const int64_t* f,
                                int64_t* dlam, int64_t* dw, int64_t* df, int32_t m,
                                int32_t n, const int32_t* order, hipStream_t st) {
  hipLaunchKernelGGL(k_gather_inputs, grid1(n, 256, 2 * m + m * m), dim3(256), 0, st, lam,
                     w, f, dlam, dw, df, m, n, order);
  return hipGetLastError();
}

hipError_t launch_gather_u8(const uint8_t* src, uint8_t* dst, int32_t rows,
                            int32_t n, const int32_t* order, hipStream_t st) {
  hipLaunchKernelGGL(k_gather_u8, grid1(n, 256, rows), dim3(256), 0, st, src,
                     dst, n, order);
  return hipGetLastError();
}

hipError_t launch_scatter_u8(const uint8_t* src, uint8_t* dst, int32_t rows,
                             int32_t n, const int32_t* order, hipStream_t st) {
  hipLaunchKernelGGL(k_scatter_u8, grid1(n, 256, rows), dim3(256), 0, st, src,
                     dst, n, order);
  return hipGetLastError();
}

hipError_t launch_scatter_i64(const int64_t* src, int64_t* dst, int32_t n,
                              const int32_t* order, hipStream_t st) {
  hipLaunchKernelGGL(k_scatter_i64, grid1(n, 256, 1), dim3(256), 0, st, src,
                     dst, n, order);
  return hipGetLastError();
}

hipError_t launch_validate(const int64_t* lam, const int64_t* w,
                           const int64_t* f, int32_t n, int32_t m,
                           uint64_t* partial, int32_t* nblocks, hipStream_t st) {
  const int64_t mn = (int64_t)m * n, mmn = mn * m;
  int64_t b = (mmn + 255) / 256;
  if (b > kValidateBlocks) b = kValidateBlocks;
  *nblocks = (int32_t)b;
  hipLaunchKernelGGL(k_validate, dim3((unsigned)b), dim3(256), 0, st, lam, w,
                     f, mn, mmn, partial);
  return hipGetLastError();
}

hipError_t launch_validate_f64(const double* lam, const double* w,
                               const double* f, int32_t n, int32_t m,
                               uint64_t* flags, int32_t* nblocks, hipStream_t st) {
  const int64_t mn = (int64_t)m * n, mmn = mn * m;
  int64_t b = (mmn + 255) / 256;
  if (b > 2 * kValidateBlocks) b = 2 * kValidateBlocks;
  *nblocks = (int32_t)b;
  hipLaunchKernelGGL(k_validate_f64, dim3((unsigned)b), dim3(256), 0, st, lam, w, f,
                     mn, mmn, flags);
  return hipGetLastError();
}

hipError_t launch_init_slots(const ChainSet& set, const DevState& d,
                             int clear_tgt, hipStream_t st) {
  int64_t mn = (int64_t)d.m * d.n;
  int64_t b = (mn + 255) / 256;
  if (b > 2048) b = 2048;
  hipLaunchKernelGGL(k_init_slots, dim3((unsigned)b, set.count), dim3(256), 0,
                     st, set, d, clear_tgt);
  return hipGetLastError();
}

hipError_t launch_holder_build(const ChainSet& set, const DevState& d,
                               hipStream_t st) {
  hipLaunchKernelGGL(k_holder_build, grid1(d.n, 256, set.count), dim3(256), 0,
                     st, set, d);
  return hipGetLastError();
}

hipError_t launch_gains(const ChainSet& set, const DevState& d, hipStream_t st,
                        int gmode, int may_skip) {
  hipLaunchKernelGGL(k_gains, grid1(d.n, 256, set.count), dim3(256), 0, st,
                     set, d, gmode, may_skip);
  return hipGetLastError();
}

hipError_t launch_assemble(const ChainSet& set, const DevState& d, int32_t dst,
                           hipStream_t st) {
  hipLaunchKernelGGL(k_assemble, grid1(d.n, 256, set.count), dim3(256), 0, st,
                     set, d, (int64_t)dst);
  return hipGetLastError();
}

hipError_t launch_mat_cost(const DevState& d, int32_t inc, int32_t prop,
                           void* partial, int32_t* nblocks, hipStream_t st) {
  int64_t b = ((int64_t)d.m * d.n + 255) / 256;
  if (b > 1024) b = 1024;
  *nblocks = (int32_t)b;
  hipLaunchKernelGGL(k_mat_cost, dim3((unsigned)b), dim3(256), 0, st, d,
                     (int64_t)inc, (int64_t)prop, (unsigned __int128*)partial);
  return hipGetLastError();
}

hipError_t launch_requester_check(const int64_t* f, int32_t n, int32_t m,
                                  int32_t* mismatch, hipStream_t st) {
  int64_t b = ((int64_t)m * n + 255) / 256;
  if (b > 1024) b = 1024;
  hipLaunchKernelGGL(k_requester_check, dim3((unsigned)b), dim3(256), 0, st, f,
                     n, m, mismatch);
  return hipGetLastError();
}

size_t dp_lds_bytes(int cells, int32_t slots_lds) {
  // control area, then the slot rows, the zero row and the sink rows
  const size_t ctl = cells == 1 ? dp_ctl_bytes<1>() : cells == 2 ? dp_ctl_bytes<2>()
                                                                 : dp_ctl_bytes<4>();
  return ctl + (size_t)(slots_lds + 1 + dp_sink_rows(cells)) * dp_row_stride(cells);
}

template <int C, bool FMAX, bool F64 = false>
static hipError_t dp_launch_c(const ChainSet& set, const DevState& d,
                              uint32_t epoch, uint32_t spin_limit,
                              int store_bits, int32_t slots_lds,
                              hipStream_t st) {
  const size_t lds = dp_lds_bytes(C, slots_lds);
  hipLaunchKernelGGL((k_dp<C, FMAX, F64>), dim3((unsigned)set.base[set.count]),
                     dim3(2 * kWave), lds, st, set, d, epoch, spin_limit,
                     store_bits, slots_lds);
  return hipGetLastError();
}

hipError_t launch_dp(const ChainSet& set, const DevState& d, uint32_t epoch,
                     uint32_t spin_limit, int store_bits, int32_t slots_lds,
                     int fmax, hipStream_t st) {
  if (d.f64) {
    // doubles: v_max_f64 is the plain maximum
    switch (d.cells) {
      case 1: return dp_launch_c<1, true, true>(set, d, epoch, spin_limit, store_bits, slots_lds, st);
      case 2: return dp_launch_c<2, true, true>(set, d, epoch, spin_limit, store_bits, slots_lds, st);
      case 4: return dp_launch_c<4, true, true>(set, d, epoch, spin_limit, store_bits, slots_lds, st);
      default: return hipErrorInvalidValue;
    }
  }
  switch (d.cells * 2 + (fmax ? 1 : 0)) {
    case 2: return dp_launch_c<1, false>(set, d, epoch, spin_limit, store_bits, slots_lds, st);
    case 3: return dp_launch_c<1, true>(set, d, epoch, spin_limit, store_bits, slots_lds, st);
    case 4: return dp_launch_c<2, false>(set, d, epoch, spin_limit, store_bits, slots_lds, st);
    case 5: return dp_launch_c<2, true>(set, d, epoch, spin_limit, store_bits, slots_lds, st);
    case 8: return dp_launch_c<4, false>(set, d, epoch, spin_limit, store_bits, slots_lds, st);
    case 9: return dp_launch_c<4, true>(set, d, epoch, spin_limit, store_bits, slots_lds, st);
    default: return hipErrorInvalidValue;
  }
}

namespace {
int dp_resident_blocks_query(int cells, int32_t slots_lds, int device);
}

// Stage blocks of the sweep that fit the device at once (occupancy queries,
// remembered per width, LDS stack height and device).
int dp_resident_blocks(int cells, int32_t slots_lds, int device) {
  static std::mutex mu;
  static std::vector<std::pair<std::array<int, 3>, int>> known;
  const std::array<int, 3> key = {cells, (int)slots_lds, device};
  {
    std::lock_guard<std::mutex> g(mu);
    for (const auto& kv : known)
      if (kv.first == key) return kv.second;
  }
  const int v = dp_resident_blocks_query(cells, slots_lds, device);
  if (v > 0) {
    std::lock_guard<std::mutex> g(mu);
    known.emplace_back(key, v);
  }
  return v;
}

namespace {
int dp_resident_blocks_query(int cells, int32_t slots_lds, int device) {
  int per_cu = 0, per_cu_f = 0, cus = 0;
  const size_t lds = dp_lds_bytes(cells, slots_lds);
  hipError_t e = hipErrorInvalidValue, e2 = hipErrorInvalidValue;
  // the integer and the real-valued variants; the smaller residency holds
  // for both
  switch (cells) {
    case 1:
      e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_dp<1, false, false>, 2 * kWave, lds);
      e2 = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu_f, k_dp<1, true, true>, 2 * kWave, lds);
      break;
    case 2:
      e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_dp<2, false, false>, 2 * kWave, lds);
      e2 = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu_f, k_dp<2, true, true>, 2 * kWave, lds);
      break;
    case 4:
      e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_dp<4, false, false>, 2 * kWave, lds);
      e2 = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu_f, k_dp<4, true, true>, 2 * kWave, lds);
      break;
    default: return 0;
  }
  if (e != hipSuccess || e2 != hipSuccess) return 0;
  per_cu = std::min(per_cu, per_cu_f);
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess)
    return 0;
  return per_cu * cus;
}
}  // namespace

hipError_t launch_backtrack(const ChainSet& set, const DevState& d, int mode,
                            hipStream_t st) {
  switch (d.cells) {
    case 1: hipLaunchKernelGGL(k_backtrack<1>, dim3(set.count), dim3(kWave), 0, st, set, d, mode); break;
    case 2: hipLaunchKernelGGL(k_backtrack<2>, dim3(set.count), dim3(kWave), 0, st, set, d, mode); break;
    case 4: hipLaunchKernelGGL(k_backtrack<4>, dim3(set.count), dim3(kWave), 0, st, set, d, mode); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_adopt(const AdoptSet& set, const DevState& d, hipStream_t st) {
  if (set.count == 0) return hipSuccess;
  hipLaunchKernelGGL(k_adopt, dim3(set.count), dim3(256), 0, st, set, d);
  return hipGetLastError();
}

hipError_t launch_take_standalone(const ChainSet& set, const DevState& d,
                                 const uint32_t* sel0, hipStream_t st) {
  if (set.count == 0) return hipSuccess;
  hipLaunchKernelGGL(k_take_standalone, dim3(set.count), dim3(256), 0, st, set, d, sel0);
  return hipGetLastError();
}

hipError_t launch_commit(const ChainSet& set, const DevState& d, int mode,
                         hipStream_t st) {
  hipLaunchKernelGGL(k_commit, grid1(d.n, kCommitThreads / d.m, set.count),
                     dim3(kCommitThreads), 0, st, set, d, mode);
  return hipGetLastError();
}

hipError_t launch_objective(const ChainSet& set, const DevState& d,
                            hipStream_t st) {
  if (d.f64) return launch_gexact(set, d, -1, st);
  int64_t mn = (int64_t)d.m * d.n;
  int64_t b = (mn + 255) / 256;
  if (b > 1024) b = 1024;
  hipLaunchKernelGGL(k_objective, dim3((unsigned)b, set.count), dim3(256), 0,
                     st, set, d);
  return hipGetLastError();
}

int32_t gexact_blocks(int32_t n, int32_t m) {
  // 128 blocks per chain, more only where a block would otherwise sum more
  // than 2^30 terms (its lazy 64-bit limbs take at most one 32-bit chunk
  // per term); never more than one block per 256 terms
  const int64_t mn = (int64_t)m * n;
  const int64_t need = (mn + (1ll << 30) - 1) >> 30;
  const int64_t b = std::min<int64_t>((mn + 255) / 256, std::max<int64_t>(128, need));
  return (int32_t)std::max<int64_t>(1, std::min<int64_t>(b, kGexactBlocks));
}

hipError_t launch_gexact(const ChainSet& set, const DevState& d, int mode,
                         hipStream_t st) {
  if (set.count == 0) return hipSuccess;
  const int32_t b = gexact_blocks(d.n, d.m);
  if (b > d.gx_blocks) return hipErrorInvalidValue;
  const int replace = (mode == kModeGreedy || mode == kModeRefine) ? 1 : 0;
  hipLaunchKernelGGL(k_gexact, dim3((unsigned)b, set.count), dim3(256), 0, st, set, d,
                     replace);
  hipLaunchKernelGGL(k_gexact_final, dim3(set.count), dim3(256), 0, st, set, d, mode,
                     (int)b);
  return hipGetLastError();
}

// ------------------------------------------- allocation-free objective --

// F_pair(T) of Eq. 6 for callers that cannot allocate device memory.  Its
// per-block partial sums live in `scratch`, one array per GPU for the life
// of the process; every call on a GPU shares it (overlapping calls on one
// GPU race), and each call writes every partial it later reads, so nothing
// needs clearing.  Layout: kNaBlocks 16-byte objective partials, kNaBlocks
// 16-byte partials of sum lam*w (overflow check), kNaBlocks 4-byte flags
// (some input negative), then the totals (NaTotals).
constexpr int kNaBlocks = 1024;

struct NaTotals {
  unsigned __int128 obj;  // sum over (r, b) of lam_r(b) * v1_r(b)
  unsigned __int128 lw;   // sum of lam * w, saturated at 2^64
  uint32_t bad;           // nonzero: a negative demand or cost
  uint32_t pad[3];
};

constexpr size_t kNaTotalsOffset = (size_t)kNaBlocks * (16 + 16 + 4);
constexpr size_t kNaScratchBytes = kNaTotalsOffset + sizeof(NaTotals);
static_assert(kNaTotalsOffset % 16 == 0, "totals alignment");
static_assert(kNaScratchBytes <= kNoAllocScratchBytes, "declared scratch size");

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

constexpr unsigned __int128 kNaSat = (unsigned __int128)1 << 64;

__device__ __forceinline__ unsigned __int128 sat_add(unsigned __int128 a,
                                                     unsigned __int128 b) {
  const unsigned __int128 s = a + b;
  return s > kNaSat ? kNaSat : s;
}

// One thread per (requester r, chunk b) in a grid-stride loop over the
// caller's layout: v1 = best saving of r over the holders of b (Eq. 5; 0 if
// none holds it), term lam_r(b) * v1; fetch costs are scanned for negative
// entries.  A held chunk is any nonzero target byte.
__global__ void __launch_bounds__(256) k_objective_na(int32_t n, int32_t m,
                                                      const int64_t* __restrict__ lam,
                                                      const int64_t* __restrict__ w,
                                                      const int64_t* __restrict__ f,
                                                      const uint8_t* __restrict__ tgt,
                                                      unsigned char* scr) {
  unsigned __int128* part_obj = (unsigned __int128*)scr;
  unsigned __int128* part_lw = part_obj + kNaBlocks;
  uint32_t* part_bad = (uint32_t*)(part_lw + kNaBlocks);
  const int64_t mn = (int64_t)m * n, mmn = mn * m;
  const int64_t step = (int64_t)gridDim.x * blockDim.x;
  unsigned __int128 acc = 0, lw = 0;
  bool bad = false;
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < mn; x += step) {
    const int r = (int)(x / n);
    const int64_t b = x % n;
    const int64_t L = lam[x], W = w[x];
    if (L < 0 || W < 0) {
      bad = true;
      continue;
    }
    int64_t v1 = 0;
    for (int l = 0; l < m; ++l) {
      if (!tgt[(int64_t)l * n + b]) continue;
      const int64_t q = l == r ? W : imax(W - f[((int64_t)l * m + r) * n + b], 0);
      v1 = imax(v1, q);
    }
    acc = sat_add(acc, (unsigned __int128)(uint64_t)L * (uint64_t)v1);
    lw = sat_add(lw, (unsigned __int128)(uint64_t)L * (uint64_t)W);
  }
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < mmn; x += step)
    if (f[x] < 0) bad = true;
  __shared__ unsigned __int128 so[256], sl[256];
  so[threadIdx.x] = acc;
  sl[threadIdx.x] = lw;
  bad = __syncthreads_or(bad);
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) {
      so[threadIdx.x] = sat_add(so[threadIdx.x], so[threadIdx.x + o]);
      sl[threadIdx.x] = sat_add(sl[threadIdx.x], sl[threadIdx.x + o]);
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    part_obj[blockIdx.x] = so[0];
    part_lw[blockIdx.x] = sl[0];
    part_bad[blockIdx.x] = bad ? 1u : 0u;
  }
}

// The totals of the first `nblocks` partials (one block).
__global__ void __launch_bounds__(256) k_objective_na_final(int32_t nblocks,
                                                            unsigned char* scr) {
  const unsigned __int128* part_obj = (const unsigned __int128*)scr;
  const unsigned __int128* part_lw = part_obj + kNaBlocks;
  const uint32_t* part_bad = (const uint32_t*)(part_lw + kNaBlocks);
  unsigned __int128 a = 0, l = 0;
  bool bad = false;
  for (int q = threadIdx.x; q < nblocks; q += blockDim.x) {
    a = sat_add(a, part_obj[q]);
    l = sat_add(l, part_lw[q]);
    bad |= part_bad[q] != 0;
  }
  __shared__ unsigned __int128 so[256], sl[256];
  so[threadIdx.x] = a;
  sl[threadIdx.x] = l;
  bad = __syncthreads_or(bad);
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) {
      so[threadIdx.x] = sat_add(so[threadIdx.x], so[threadIdx.x + o]);
      sl[threadIdx.x] = sat_add(sl[threadIdx.x], sl[threadIdx.x + o]);
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    NaTotals* t = (NaTotals*)(scr + kNaTotalsOffset);
    t->obj = so[0];
    t->lw = sl[0];
    t->bad = bad ? 1u : 0u;
  }
}

}  // namespace

// Device address of `scratch` on each GPU, looked up once per device with
// that device current (each GPU holds its own copy of the array).
static void* g_na_ptr[kNoAllocMaxDevices];
static std::mutex g_na_mu;

hipError_t noalloc_scratch(int device, void** ptr) {
  if (device < 0 || device >= kNoAllocMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_na_mu);
  if (!g_na_ptr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_na_ptr[device] = p;
  }
  *ptr = g_na_ptr[device];
  return hipSuccess;
}

hipError_t launch_objective_noalloc(int32_t n, int32_t m, const int64_t* lam,
                                    const int64_t* w, const int64_t* f,
                                    const uint8_t* tgt, void* scr,
                                    NoAllocResult* out, hipStream_t st) {
  const int64_t mn = (int64_t)m * n;
  int64_t b = (mn + 255) / 256;
  if (b > kNaBlocks) b = kNaBlocks;
  if (b < 1) b = 1;
  unsigned char* s = (unsigned char*)scr;
  hipLaunchKernelGGL(k_objective_na, dim3((unsigned)b), dim3(256), 0, st, n, m,
                     lam, w, f, tgt, s);
  hipLaunchKernelGGL(k_objective_na_final, dim3(1), dim3(256), 0, st, (int32_t)b, s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  NaTotals t;
  e = hipMemcpyAsync(&t, s + kNaTotalsOffset, sizeof t, hipMemcpyDeviceToHost, st);
  if (e != hipSuccess) return e;
  e = hipStreamSynchronize(st);
  if (e != hipSuccess) return e;
  out->bad = t.bad != 0;
  out->overflow = t.lw > (unsigned __int128)INT64_MAX;
  out->objective = out->overflow ? 0 : (int64_t)t.obj;
  return hipSuccess;
}

}  // namespace pp
