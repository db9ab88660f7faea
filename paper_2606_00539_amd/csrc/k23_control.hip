// K2 and K3 of the GNMR controller pass for CDNA4 (gfx950).
//
//   K2 k2_update   per unit: fixed-order float64 sum of its K1 partials,
//                  n = sqrt, then Alg. 1 (GNMR, Delta-GNMR, running mean,
//                  queue), the risk R of Alg. 2, and membership of the
//                  candidate pool C_t (Alg. 2; Sec. 3.3)
//   K3 k3_select   one workgroup: Top_maxO over C_t by R (ties to the smaller
//                  index), lock update and step counters (Alg. 2; Sec. 3.3,
//                  3.4)
//
// Deterministic: fixed reduction orders, integer atomics only.
#include <math.h>

#include "gnmr_internal.h"

namespace gnmr {
namespace {

// Butterfly over the 64 lanes of a wavefront; every lane ends with the same sum.
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// Fixed-order float64 sum of unit b's item partials by L lanes (lane < L):
// each lane keeps four running sums over a stride-L walk, then the lanes are
// combined by a fixed butterfly (L = 64) and a fixed cross-wave order
// (L = 256).  L = 1 is one thread per unit, for units of few items.
template <int L>
__device__ __forceinline__ double unit_ss(const int64_t* __restrict__ off,
                                          const float* __restrict__ partial, int b, int lane,
                                          double* red) {
  double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
  const int64_t hi = off[b + 1];
  int64_t i = off[b] + lane;
  for (; i + 3 * L < hi; i += 4 * L) {
    const float a = partial[i], c = partial[i + L], d = partial[i + 2 * L], e = partial[i + 3 * L];
    s0 += double(a);
    s1 += double(c);
    s2 += double(d);
    s3 += double(e);
  }
  for (; i < hi; i += L) s0 += double(partial[i]);
  const double s = (s0 + s1) + (s2 + s3);
  if constexpr (L == 1) {
    return s;
  } else if constexpr (L == 64) {
    return wave_sum(s);
  } else {
    static_assert(L == 256, "1, 64 or 256 lanes per unit");
    const double w = wave_sum(s);
    if ((lane & 63) == 0) red[lane >> 6] = w;
    __syncthreads();
    return ((red[0] + red[1]) + red[2]) + red[3];
  }
}

template <int L>
__global__ __launch_bounds__(256) void k_unit_sumsq(const int64_t* __restrict__ off,
                                                    const float* __restrict__ partial,
                                                    int num_units, double* __restrict__ out) {
  __shared__ double red[4];
  const int lane = L == 1 ? 0 : int(threadIdx.x % L);
  const int b = blockIdx.x * (256 / L) + threadIdx.x / L;
  if (b >= num_units) return;  // uniform per workgroup when L = 256
  const double s = unit_ss<L>(off, partial, b, lane, red);
  if (lane == 0) out[b] = s;
}

// n_{b,t} from a unit's float64 sum of squares.  The sums of squares are
// accumulated in fp32, whose range ends at 2^128: a unit whose sum reaches it
// (a gradient norm of 2^64 or more) has no representable fp32 sum, so its
// norm is taken as +inf, a non-finite norm (the outcome when an fp32 square
// or partial overflows, made independent of how the sum is split into items).
// NaN stays NaN.
__device__ __forceinline__ double norm_of_sumsq(double ss) {
  return ss >= 0x1p128 ? double(INFINITY) : sqrt(ss);
}

// Order-preserving key of a candidate: R >= 0 (or +inf), so its IEEE bits
// are monotone in R; +1 keeps 0 free for "not a candidate".
__device__ __forceinline__ uint64_t cand_key(double R) {
  return uint64_t(__double_as_longlong(R)) + 1;
}

// What one unit adds to the step's counters and candidate list.
struct Contrib {
  bool cand, ranked, tg, td, tr, nonfinite;
};

// Alg. 1 and the risk of Alg. 2 for unit b given its norm n, and the unit's
// membership of the candidate pool C_t; returns what it adds to the counters.
__device__ __forceinline__ Contrib update_unit(const UpdateArgs& a, int b, double n) {
  const int U = a.num_units;
  // The step counter lives on the device, so that a captured step replays
  // correctly: t = 1 + steps completed, the queue holds min(t - 1, delta)
  // values, and the oldest value sits in the slot the new one replaces.
  const int64_t t = *a.step + 1;
  const int qlen = t - 1 < a.window ? int(t - 1) : a.window;
  const int slot0 = int((t - 1) % a.window);
  const bool warm = t <= a.warmup;
  const bool finite = isfinite(n);
  const double A_prev = a.A[b];
  // Alg. 1: GNMR = 1 at t = 1 or while the historical mean is 0.
  double G = 1.0;
  if (finite && t > 1 && A_prev != 0.0) G = n / (A_prev + a.eps);
  // Alg. 1: Delta-GNMR once the queue holds delta values, oldest first.
  double D = 1.0;
  if (qlen == a.window) {
    double total = 0.0;
    int slot = slot0;
    for (int j = 0; j < a.window; ++j) {
      total += a.Q[int64_t(slot) * U + b];
      slot = slot + 1 == a.window ? 0 : slot + 1;
    }
    const double den = total / double(a.window) + a.eps;
    if (finite && den != 0.0) D = G / den;
  }
  // Alg. 1: running mean and queue push (the new value replaces the oldest).
  if (finite) a.A[b] = A_prev + (n - A_prev) / double(t);
  a.Q[int64_t(slot0) * U + b] = finite ? G : 1.0;
  if (!finite) G = D = INFINITY;

  // Alg. 2: R = max(GNMR / alpha, Delta-GNMR / beta); the pool C_t holds the
  // recoverable units with R > 1 or a lock left from the previous step.
  const double gt = G / a.alpha;
  const double dt = D / a.beta;
  const double R = gt > dt ? gt : dt;
  const bool rec = a.rec[b] != 0;
  const bool trig = R > 1.0;
  bool cand = rec && (trig || a.lock[b] > 0);
  bool keep = false;
  double rank_by = R;
  if (a.static_set) {                 // static baseline: profile, rank once, hold
    if (t <= a.warmup) {
      a.gsum[b] += finite ? G : 0.0;
      cand = keep = rec;
    } else if (t == a.warmup + 1) {
      cand = rec;
      rank_by = a.gsum[b] / double(a.warmup);   // mean GNMR over steps 1..W
    } else {
      cand = keep = a.mask[b] != 0;
    }
  } else if (warm) {                  // warm-up: C_t = A_t = B_rec
    cand = rec;
    keep = rec;
  } else if (a.admitted && cand) {    // admitted-only budget: A_{t-1} members stay
    keep = a.mask[b] != 0;
  }
  const bool ranked = cand && !keep;
  const bool tg = rec && gt > 1.0, td = rec && dt > 1.0, tr = rec && trig;
  a.norm[b] = n;
  a.gnmr[b] = G;
  a.dgnmr[b] = D;
  a.risk[b] = R;
  a.keys[b] = ranked ? cand_key(rank_by) : 0;
  a.flags[b] = uint8_t((gt > 1.0 ? kFlagTrigG : 0) | (dt > 1.0 ? kFlagTrigD : 0) |
                       (finite ? 0 : kFlagNonFinite) | (trig ? kFlagTrigR : 0) |
                       (rec ? kFlagRec : 0) | (cand ? kFlagCand : 0) |
                       (keep ? kFlagKeep : 0));
  // Alg. 2 outcome of a unit outside C_t is fixed already: low-cost path,
  // Lock = 0.  K3 only has to rank and update the members of C_t.
  if (!cand) {
    a.mask[b] = 0;
    if (a.lock[b] != 0) a.lock[b] = 0;
  }
  return Contrib{cand, ranked, tg, td, tr, !finite};
}

// Adds the contributions of a workgroup's units (`has`: this thread holds
// unit b) to counter set blockIdx.x % kCounterSets and appends its members
// of C_t to that set's list: summed by ballot and LDS first, then one global
// atomic per counter and workgroup (integer atomics: exact; the list order
// is irrelevant to the selection).  Called by every thread of the workgroup.
__device__ void publish(const UpdateArgs& a, bool has, int b, const Contrib& c) {
  __shared__ int32_t s_cnt[kNumCounters];
  __shared__ int32_t s_base;
  const int tid = int(threadIdx.x), wl = tid & 63;
  if (tid < kNumCounters) s_cnt[tid] = 0;
  __syncthreads();
  const uint64_t m_c = __ballot(has && c.cand);
  const uint64_t m_k = __ballot(has && c.ranked), m_g = __ballot(has && c.tg);
  const uint64_t m_d = __ballot(has && c.td), m_r = __ballot(has && c.tr);
  const uint64_t m_n = __ballot(has && c.nonfinite);
  int wave_base = 0;
  if (wl == 0) {
    if (m_c) wave_base = atomicAdd(&s_cnt[kCntCand], __popcll(m_c));
    if (m_k) atomicAdd(&s_cnt[kCntRank], __popcll(m_k));
    if (m_g) atomicAdd(&s_cnt[kCntTrigG], __popcll(m_g));
    if (m_d) atomicAdd(&s_cnt[kCntTrigD], __popcll(m_d));
    if (m_r) atomicAdd(&s_cnt[kCntTrigR], __popcll(m_r));
    if (m_n) atomicAdd(&s_cnt[kCntNonFinite], __popcll(m_n));
  }
  wave_base = __shfl(wave_base, 0, 64);
  const int slot = wave_base + __popcll(m_c & ((uint64_t(1) << wl) - 1));
  __syncthreads();
  const int set = int(blockIdx.x % kCounterSets);
  if (tid == 0) {
    int32_t* cs = a.counters + set * kNumCounters;
    s_base = s_cnt[kCntCand] ? atomicAdd(&cs[kCntCand], s_cnt[kCntCand]) : 0;
#pragma unroll
    for (int k = 1; k < kNumCounters; ++k)
      if (s_cnt[k]) atomicAdd(&cs[k], s_cnt[k]);
  }
  __syncthreads();
  if (has && c.cand) a.cand_list[set * a.list_cap + s_base + slot] = b;
}

// The same for a kernel of one workgroup whose counters and list are in LDS:
// one LDS atomic per counter and wavefront, no barrier (the caller's next
// barrier makes the results visible).
__device__ __forceinline__ void publish_local(int32_t* cnt, int32_t* list, bool has, int b,
                                              const Contrib& c) {
  const int wl = int(threadIdx.x & 63);
  const uint64_t m_c = __ballot(has && c.cand);
  const uint64_t m_k = __ballot(has && c.ranked), m_g = __ballot(has && c.tg);
  const uint64_t m_d = __ballot(has && c.td), m_r = __ballot(has && c.tr);
  const uint64_t m_n = __ballot(has && c.nonfinite);
  int base = 0;
  if (wl == 0) {
    if (m_c) base = atomicAdd(&cnt[kCntCand], __popcll(m_c));
    if (m_k) atomicAdd(&cnt[kCntRank], __popcll(m_k));
    if (m_g) atomicAdd(&cnt[kCntTrigG], __popcll(m_g));
    if (m_d) atomicAdd(&cnt[kCntTrigD], __popcll(m_d));
    if (m_r) atomicAdd(&cnt[kCntTrigR], __popcll(m_r));
    if (m_n) atomicAdd(&cnt[kCntNonFinite], __popcll(m_n));
  }
  base = __shfl(base, 0, 64);
  if (has && c.cand) list[base + __popcll(m_c & ((uint64_t(1) << wl) - 1))] = b;
}

// K2: L lanes per unit sum its partials; lane 0 then runs Alg. 1, the risk of
// Alg. 2, and marks the unit's membership of the candidate pool C_t.
template <int L>
__global__ __launch_bounds__(256) void k2_update(UpdateArgs a) {
  __shared__ double red[4];
  const int lane = L == 1 ? 0 : int(threadIdx.x % L);
  const int b = blockIdx.x * (256 / L) + threadIdx.x / L;
  if (L == 256 && b >= a.num_units) return;  // the whole workgroup
  const bool in = b < a.num_units;           // uniform per wavefront when L = 64
  double n = 0.0;
  if (in) {
    if (a.ext_norm != nullptr) {
      n = a.ext_norm[b];
    } else {
      n = norm_of_sumsq(unit_ss<L>(a.unit_item_off, a.partial, b, lane, red));
    }
  }
  const bool has = in && lane == 0;
  Contrib c{};
  if (has) c = update_unit(a, b, n);
  publish(a, has, b, c);
}

constexpr int kK3Block = 1024;
constexpr int kK3Cap = 12288;  // candidates held in LDS (144 KiB); larger pools use the global keys
constexpr int kK3Count = 128;  // pools up to this size are ranked by direct counting

// Lock update of Alg. 2 for one unit given its selection.
__device__ __forceinline__ void apply_selection(const SelectArgs& a, int b, bool sel, uint8_t f) {
  int32_t L = 0;
  if (sel) {
    const int32_t prev = a.lock[b];
    L = (f & kFlagTrigR) ? a.lock_len : (prev > 0 ? prev - 1 : 0);
  }
  a.lock[b] = L;
  a.mask[b] = sel ? 1 : 0;
}

// MSB-first radix select, 8 passes of 8 bits: the k-th largest (1-based) of
// the n keys key_at(i), i < n.  Returns it as T; *rest receives how many keys
// equal to T are among the k largest.  Called by every thread of the
// workgroup.  Two barriers per pass: the histograms alternate between the
// two halves of hist[512], so a pass clears the next pass's half (last read
// before the previous pass's second barrier) while it counts into its own,
// and the digit it publishes is read by every thread before any thread can
// reach the barrier after which the next digit is written.
//
// Once the bucket that holds the k-th largest key has at most 64 keys, the
// passes stop: those keys are gathered into LDS and one wavefront finishes by
// counting, for each, the keys above it (a typical pool of a few thousand R
// values gets there after 3 of the 8 passes).
struct RadixSmall {
  uint64_t key[64];
  int n;                  // keys gathered
  int bucket;             // keys in the chosen bucket (written with the digit)
  uint64_t T;
  int rest;
};

template <typename KeyAt>
__device__ uint64_t radix_select(KeyAt key_at, int n, int k, uint32_t* hist, int* s_digit,
                                 int* s_k, int* rest, RadixSmall* sm) {
  const int tid = threadIdx.x;
  uint64_t prefix = 0, pmask = 0;
  if (tid < 256) hist[tid] = 0;
  __syncthreads();
  for (int shift = 56, pass = 0; shift >= 0; shift -= 8, ++pass) {
    uint32_t* const h = hist + (pass & 1) * 256;
    if (tid < 256) hist[((pass + 1) & 1) * 256 + tid] = 0;
    if (tid == 0) sm->n = 0;
    // In the upper bytes of R's bits the keys of a wavefront mostly share
    // one digit: then one lane adds them all (one LDS atomic, not one per key
    // on the same counter); otherwise every key adds itself.
    const int rounds = (n + kK3Block - 1) / kK3Block;
    for (int r = 0; r < rounds; ++r) {
      const int i = tid + r * kK3Block;
      bool pend = false;
      uint32_t d = 0;
      if (i < n) {
        const uint64_t key = key_at(i);
        pend = (key & pmask) == prefix;
        d = uint32_t(key >> shift) & 255u;
      }
      const uint64_t m = __ballot(pend);
      if (m == 0) continue;
      const int leader = __ffsll((unsigned long long)m) - 1;
      const uint32_t dl = __shfl(d, leader, 64);
      if (__ballot(pend && d == dl) == m) {
        if ((tid & 63) == leader) atomicAdd(&h[dl], uint32_t(__popcll(m)));
      } else if (pend) {
        atomicAdd(&h[d], 1u);
      }
    }
    __syncthreads();
    if (tid < 64) {
      // The digit of the k-th largest key: the largest d whose count of keys
      // with a digit above d is below k, found by one wavefront: lane l holds
      // digits 4l .. 4l+3, a suffix sum over the lanes gives the count above
      // each lane's digits, and the one lane whose digits reach k names d
      // (k <= the keys in the histogram, so exactly one lane does).
      const int l = tid;
      const uint32_t h0 = h[4 * l], h1 = h[4 * l + 1], h2 = h[4 * l + 2], h3 = h[4 * l + 3];
      const uint32_t own = h0 + h1 + h2 + h3;
      uint32_t suffix = own;  // keys with a digit >= 4l
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t v = __shfl_down(suffix, off, 64);
        if (l + off < 64) suffix += v;
      }
      uint32_t above = suffix - own;  // keys with a digit above 4l+3
      const uint32_t uk = uint32_t(k);
      if (above < uk && above + own >= uk) {
        int d = 4 * l + 3;
        const uint32_t hv[4] = {h0, h1, h2, h3};
        for (int j = 3; j > 0 && above + hv[j] < uk; --j, --d) above += hv[j];
        *s_digit = d;
        *s_k = k - int(above);
        sm->bucket = int(d == 4 * l + 3 ? h3 : d == 4 * l + 2 ? h2 : d == 4 * l + 1 ? h1 : h0);
      }
    }
    __syncthreads();
    prefix |= uint64_t(*s_digit) << shift;
    pmask |= uint64_t(255) << shift;
    k = *s_k;
    if (shift > 0 && sm->bucket <= 64) {
      // gather the bucket (prefix matched so far) and finish by counting
      for (int i = tid; i < n; i += kK3Block) {
        const uint64_t key = key_at(i);
        if ((key & pmask) == prefix) sm->key[atomicAdd(&sm->n, 1)] = key;
      }
      __syncthreads();
      if (tid < 64) {
        const int m = sm->n;
        const uint64_t mine = tid < m ? sm->key[tid] : 0;
        int above = 0, not_below = 0;
        for (int j = 0; j < m; ++j) {
          const uint64_t kj = sm->key[j];
          above += kj > mine ? 1 : 0;
          not_below += kj >= mine ? 1 : 0;
        }
        // the k-th largest: fewer than k keys above it, at least k at or above
        if (tid < m && above < k && not_below >= k) {
          sm->T = mine;
          sm->rest = k - above;
        }
      }
      __syncthreads();
      *rest = sm->rest;
      return sm->T;
    }
  }
  *rest = k;
  return prefix;
}

// Selection over every unit from the global keys: kept units, key > T, or
// key == T and among the first `need` such units in index order (contiguous
// index ranges per thread and an exclusive scan of their tie counts).
__device__ int select_by_scan(const SelectArgs& a, uint64_t T, int need, uint32_t* scan) {
  const int tid = threadIdx.x;
  const int U = a.num_units;
  const int per = (U + kK3Block - 1) / kK3Block;
  const int lo = tid * per < U ? tid * per : U;
  const int hi = lo + per < U ? lo + per : U;
  uint32_t ties = 0;
  for (int b = lo; b < hi; ++b) ties += a.keys[b] == T;
  scan[tid] = ties;
  __syncthreads();
  for (int d = 1; d < kK3Block; d <<= 1) {
    const uint32_t v = tid >= d ? scan[tid - d] : 0;
    __syncthreads();
    scan[tid] += v;
    __syncthreads();
  }
  uint32_t rank = scan[tid] - ties;  // ties before this thread's range
  int c_act = 0;
  for (int b = lo; b < hi; ++b) {
    const uint64_t key = a.keys[b];
    const uint8_t f = a.flags[b];
    bool sel = key > T;
    if (key == T) {
      sel = rank < uint32_t(need);
      ++rank;
    }
    sel = sel || (f & kFlagKeep);
    apply_selection(a, b, sel, f);
    c_act += sel;
  }
  return c_act;
}

// Ascending bitonic sort of v[0..kK3Block) in LDS by the whole workgroup.
__device__ void bitonic_sort(int32_t* v) {
  const int tid = threadIdx.x;
  for (int size = 2; size <= kK3Block; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      __syncthreads();
      const int j = tid ^ stride;
      if (j > tid) {
        const bool up = (tid & size) == 0;
        const int32_t x = v[tid], y = v[j];
        if ((x > y) == up) {
          v[tid] = y;
          v[j] = x;
        }
      }
    }
  }
  __syncthreads();
}

// K3: a single workgroup, over the members of C_t listed by K2.  Kept units
// (warm-up; continuing units under the admitted-only budget) are active
// without ranking; the others are ranked for the budget.  When at most maxO
// are ranked they are all active.  Otherwise small pools (up to kK3Count)
// count each candidate's place in the order directly; larger ones need the
// maxO-th largest ranked key T (radix select; kept units carry
// key 0): every ranked candidate with key > T is active, and the first
// `need` with key == T in index order.  Pools of up to kCap candidates are
// ranked in LDS; larger ones over the global keys of all units.
template <int kCap>
__device__ void select_body(const SelectArgs& a) {
  __shared__ uint64_t c_key[kCap];
  __shared__ int32_t c_idx[kCap];
  __shared__ int32_t tie_idx[kK3Block];
  __shared__ uint32_t hist[2 * 256];
  __shared__ RadixSmall rsm;
  __shared__ int cnt[2];  // active, ties
  __shared__ int s_digit, s_k;
  uint32_t* scan = reinterpret_cast<uint32_t*>(tie_idx);  // the global path reuses it
  const int tid = threadIdx.x;
  const int U = a.num_units;
  // Gather K2's counter sets: totals, and where each set's candidates start
  // in the pool's order (one thread per counter, then one for the offsets).
  __shared__ int32_t s_sets[kCounterSets * kNumCounters];
  __shared__ int32_t s_tot[kNumCounters];
  __shared__ int32_t s_setoff[kCounterSets + 1];
  if (tid < 2) cnt[tid] = 0;
  if (a.num_sets == 1) {  // the single-workgroup kernel: one set, nothing to combine
    if (tid < kNumCounters) s_tot[tid] = a.counters[tid];
    if (tid == kNumCounters) {
      s_setoff[0] = 0;
      s_setoff[1] = a.counters[kCntCand];
    }
  } else {  // (num_sets is the same for the whole workgroup)
    if (tid < a.num_sets * kNumCounters) s_sets[tid] = a.counters[tid];
    __syncthreads();
    if (tid < kNumCounters) {
      int32_t t = 0;
      for (int j = 0; j < a.num_sets; ++j) t += s_sets[j * kNumCounters + tid];
      s_tot[tid] = t;
    } else if (tid == kNumCounters) {
      int32_t t = 0;
      s_setoff[0] = 0;
      for (int j = 0; j < a.num_sets; ++j) {
        t += s_sets[j * kNumCounters + kCntCand];
        s_setoff[j + 1] = t;
      }
    }
  }
  __syncthreads();
  const int n_cand = s_tot[kCntCand];
  const int n_rank = s_tot[kCntRank];
  // the i-th candidate of the pool: set j with s_setoff[j] <= i < s_setoff[j+1]
  auto cand_at = [&](int i) {
    int lo = 0, hi = a.num_sets;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (s_setoff[mid] <= i) lo = mid; else hi = mid;
    }
    return a.cand_list[lo * a.list_cap + (i - s_setoff[lo])];
  };

  int c_act = 0;
  if (a.max_o == 0 || n_rank <= a.max_o) {
    // no ranking: every listed unit is active, or only the kept ones if maxO = 0
    const bool take = a.max_o > 0;
    for (int i = tid; i < n_cand; i += kK3Block) {
      const int b = cand_at(i);
      const uint8_t f = a.flags[b];
      const bool sel = take || (f & kFlagKeep);
      apply_selection(a, b, sel, f);
      c_act += sel;
    }
  } else if (n_cand <= kK3Count) {
    // A small pool: each ranked candidate's place in the order (R
    // descending, index ascending) is counted directly against the whole
    // pool, one barrier instead of the radix passes.  Kept units carry key
    // 0, below every ranked key, so they never push a ranked one down; a
    // ranked candidate is active when fewer than maxO candidates come before
    // it.
    if (tid < n_cand) {
      const int b = cand_at(tid);
      c_idx[tid] = b;
      c_key[tid] = a.keys[b];
    }
    __syncthreads();
    if (tid < n_cand) {
      const int b = c_idx[tid];
      const uint64_t key = c_key[tid];
      int before = 0;
#pragma unroll 8
      for (int j = 0; j < n_cand; ++j) {
        const uint64_t kj = c_key[j];
        before += (kj > key || (kj == key && c_idx[j] < b)) ? 1 : 0;
      }
      const uint8_t f = a.flags[b];
      const bool sel = (key != 0 && before < a.max_o) || (f & kFlagKeep);
      apply_selection(a, b, sel, f);
      c_act += sel;
    }
  } else if (n_cand > kCap) {
    int need = 0;
    const uint64_t* __restrict__ keys = a.keys;
    const uint64_t T = radix_select([=](int i) { return keys[i]; }, U, a.max_o, hist, &s_digit,
                                    &s_k, &need, &rsm);
    c_act = select_by_scan(a, T, need, scan);
  } else {
    for (int i = tid; i < n_cand; i += kK3Block) {
      const int b = cand_at(i);
      c_idx[i] = b;
      c_key[i] = a.keys[b];
    }
    __syncthreads();
    int need = 0;
    const uint64_t T = radix_select([&](int i) { return c_key[i]; }, n_cand, a.max_o, hist,
                                    &s_digit, &s_k, &need, &rsm);
    // Ties at T: gather their indices; when more tie than may be taken, keep
    // the `need` smallest indices, i.e. every tie with index <= cut.
    for (int i = tid; i < n_cand; i += kK3Block) {
      if (c_key[i] == T) {
        const int slot = atomicAdd(&cnt[1], 1);
        if (slot < kK3Block) tie_idx[slot] = c_idx[i];
      }
    }
    __syncthreads();
    const int n_ties = cnt[1];
    if (n_ties > kK3Block) {
      c_act = select_by_scan(a, T, need, scan);
    } else {
      int32_t cut = INT32_MAX;  // every tie taken
      if (n_ties > need) {
        if (tid >= n_ties) tie_idx[tid] = INT32_MAX;
        bitonic_sort(tie_idx);
        cut = tie_idx[need - 1];
      }
      for (int i = tid; i < n_cand; i += kK3Block) {
        const int b = c_idx[i];
        const uint64_t key = c_key[i];
        const uint8_t f = a.flags[b];
        const bool sel = key > T || (key == T && b <= cut) || (f & kFlagKeep);
        apply_selection(a, b, sel, f);
        c_act += sel;
      }
    }
  }
  if (c_act) atomicAdd(&cnt[0], c_act);
  __syncthreads();
  if (tid == 0) {
    const int64_t t = *a.step + 1;
    const bool warm = t <= a.warmup;
    gnmr_stats st;
    st.t = t;
    st.n_trig_gnmr = s_tot[kCntTrigG];
    st.n_trig_dgnmr = s_tot[kCntTrigD];
    st.n_trig = s_tot[kCntTrigR];
    st.n_cand = n_cand;
    st.n_active = cnt[0];
    st.hit_maxo = (!warm && n_rank > 0 && n_rank >= a.max_o) ? 1 : 0;
    st.n_nonfinite = s_tot[kCntNonFinite];
    st.reserved = 0;
    *a.stats = st;
    *a.step = t;
  }
  // the counter sets, ready for the next step (read only in the gather above)
  for (int k = tid; k < a.num_sets * kNumCounters; k += kK3Block) a.counters[k] = 0;
}

__global__ __launch_bounds__(kK3Block) void k3_select(SelectArgs a) { select_body<kK3Cap>(a); }

// K2 and K3 in one workgroup, for small workloads: at most kK3Block units,
// each summed by one thread exactly as k2_update<1> sums it (or given its
// norm), then the selection of K3 after a workgroup barrier, which makes
// K2's keys and flags visible to every thread.  The counters and the
// candidate list live in LDS here (one workgroup uses them), which keeps
// global atomics off the path.  One launch instead of two; the same
// arithmetic, so the same results.
__global__ __launch_bounds__(kK3Block) void k23_small(UpdateArgs u, SelectArgs s) {
  __shared__ int32_t s_counters[kNumCounters];
  __shared__ int32_t s_cand[kK3Block];
  if (threadIdx.x < kNumCounters) s_counters[threadIdx.x] = 0;
  // one counter set, in LDS
  u.counters = s.counters = s_counters;
  u.cand_list = s_cand;
  s.cand_list = s_cand;
  u.list_cap = s.list_cap = kK3Block;
  s.num_sets = 1;
  __syncthreads();
  const int b = int(threadIdx.x);
  const bool has = b < u.num_units;
  Contrib c{};
  if (has) {
    const double n = u.ext_norm != nullptr
                         ? u.ext_norm[b]
                         : norm_of_sumsq(unit_ss<1>(u.unit_item_off, u.partial, b, 0, nullptr));
    c = update_unit(u, b, n);
  }
  publish_local(s_counters, s_cand, has, b, c);
  __syncthreads();
  select_body<kK3Block>(s);  // at most kK3Block units, so the pool fits
}

}  // namespace

// Lanes per unit for the partial sums: one thread when units have few items,
// a wavefront for moderate counts, a whole workgroup once long strided walks
// would be latency bound.
static int lanes_per_unit(int64_t num_items, int32_t num_units) {
  const int64_t per = num_items / (num_units > 0 ? num_units : 1);
  return per < 32 ? 1 : per < 512 ? 64 : 256;
}

template <int L>
static dim3 unit_grid(int32_t num_units) {
  return dim3(unsigned((int64_t(num_units) * L + 255) / 256));
}

hipError_t launch_unit_sumsq(const int64_t* unit_item_off, const float* partial,
                             int64_t num_items, int32_t num_units, double* out, hipStream_t s) {
  switch (lanes_per_unit(num_items, num_units)) {
    case 1:
      hipLaunchKernelGGL(k_unit_sumsq<1>, unit_grid<1>(num_units), dim3(256), 0, s,
                         unit_item_off, partial, num_units, out);
      break;
    case 64:
      hipLaunchKernelGGL(k_unit_sumsq<64>, unit_grid<64>(num_units), dim3(256), 0, s,
                         unit_item_off, partial, num_units, out);
      break;
    default:
      hipLaunchKernelGGL(k_unit_sumsq<256>, unit_grid<256>(num_units), dim3(256), 0, s,
                         unit_item_off, partial, num_units, out);
  }
  return hipGetLastError();
}

hipError_t launch_update(const UpdateArgs& a, int64_t num_items, hipStream_t s) {
  const int L = a.ext_norm != nullptr ? 1 : lanes_per_unit(num_items, a.num_units);
  if (L == 1)
    hipLaunchKernelGGL(k2_update<1>, unit_grid<1>(a.num_units), dim3(256), 0, s, a);
  else if (L == 64)
    hipLaunchKernelGGL(k2_update<64>, unit_grid<64>(a.num_units), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(k2_update<256>, unit_grid<256>(a.num_units), dim3(256), 0, s, a);
  return hipGetLastError();
}

bool single_launch_update_select(const UpdateArgs& a, int64_t num_items) {
  return a.num_units <= kK3Block &&
         (a.ext_norm != nullptr || lanes_per_unit(num_items, a.num_units) == 1);
}

hipError_t launch_update_select(const UpdateArgs& u, const SelectArgs& s, hipStream_t st) {
  hipLaunchKernelGGL(k23_small, dim3(1), dim3(kK3Block), 0, st, u, s);
  return hipGetLastError();
}

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k3_select, dim3(1), dim3(kK3Block), 0, s, a);
  return hipGetLastError();
}

}  // namespace gnmr
