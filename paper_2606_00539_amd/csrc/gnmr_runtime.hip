// Host runtime of libgnmr: context, argument checks, the K1 work list,
// kernel launches, outputs, state blob and kernel timing.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <array>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "gnmr_internal.h"

using gnmr::Item;

namespace {

thread_local std::string g_last_error;

gnmr_status fail(gnmr_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

#define GNMR_HIP(expr)                                                                 \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess)                                                              \
      return fail(GNMR_E_HIP, std::string(#expr) + ": " + hipGetErrorString(e_));      \
  } while (0)

constexpr uint32_t kStateMagic = 0x524D4E47u;  // "GNMR"
constexpr uint32_t kStateVersion = 4;
constexpr int kProfileCapacity = 4096;

struct StateHeader {
  uint32_t magic;
  uint32_t version;
  int32_t num_units;
  int32_t window;
  int64_t t;
  int32_t max_o;
  int32_t lock_len;
  double eps;
  int32_t budget_mode;
  int32_t warmup_steps;
};
static_assert(sizeof(StateHeader) == 48, "state header layout");

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Makes the context's device current for the duration of a call.
struct DeviceGuard {
  int prev = -1;
  bool ok = true;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) {
      ok = false;
      return;
    }
    if (prev != dev && hipSetDevice(dev) != hipSuccess) ok = false;
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

// A byte range [lo, hi) of device memory that buffer `id` covers.
struct Span {
  uintptr_t lo, hi;
  int64_t id;
};

Span span_of(const void* p, int64_t bytes, int64_t id) {
  const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
  return Span{lo, lo + uintptr_t(bytes), id};
}

bool intersect(const Span& a, const Span& b) {
  return a.lo < a.hi && b.lo < b.hi && a.lo < b.hi && b.lo < a.hi;
}

// Index of a write that overlaps another write, or a read of a different id;
// -1 when there is none.  O((W + R) log R): reads sorted by start, with the
// two largest ends of distinct ids over every prefix.
int64_t find_overlap(std::vector<Span> w, std::vector<Span> r) {
  auto by_lo = [](const Span& a, const Span& b) { return a.lo < b.lo; };
  w.erase(std::remove_if(w.begin(), w.end(), [](const Span& s) { return s.lo >= s.hi; }), w.end());
  r.erase(std::remove_if(r.begin(), r.end(), [](const Span& s) { return s.lo >= s.hi; }), r.end());
  std::sort(w.begin(), w.end(), by_lo);
  uintptr_t reach = 0;
  for (size_t k = 0; k < w.size(); ++k) {
    if (k > 0 && w[k].lo < reach) return w[k].id;
    reach = std::max(reach, w[k].hi);
  }
  std::sort(r.begin(), r.end(), by_lo);
  struct Top2 {
    uintptr_t hi1 = 0, hi2 = 0;
    int64_t id1 = -1, id2 = -1;
  };
  std::vector<Top2> pre(r.size() + 1);
  for (size_t k = 0; k < r.size(); ++k) {
    Top2 t = pre[k];
    const Span& s = r[k];
    if (s.id == t.id1) {
      t.hi1 = std::max(t.hi1, s.hi);
    } else if (t.id1 < 0 || s.hi > t.hi1) {
      t.hi2 = t.hi1;
      t.id2 = t.id1;
      t.hi1 = s.hi;
      t.id1 = s.id;
    } else if (t.id2 < 0 || s.hi > t.hi2) {
      t.hi2 = s.hi;
      t.id2 = s.id;
    }
    pre[k + 1] = t;
  }
  for (const Span& s : w) {
    // reads starting before the write ends; the furthest-reaching one of another id
    const size_t k = size_t(std::lower_bound(r.begin(), r.end(), Span{s.hi, s.hi, 0}, by_lo) -
                            r.begin());
    const Top2& t = pre[k];
    const bool other1 = t.id1 >= 0 && t.id1 != s.id;
    const uintptr_t hi = other1 ? t.hi1 : (t.id2 >= 0 ? t.hi2 : 0);
    if ((other1 || t.id2 >= 0) && hi > s.lo) return s.id;
  }
  return -1;
}

}  // namespace

struct gnmr_ctx {
  int device = 0;
  int32_t U = 0, window = 0, max_o = 0, lock_len = 0;
  int32_t budget_mode = GNMR_BUDGET_ACTIVE, warmup_steps = 0;
  double eps = 0.0;
  int64_t S = 0;
  std::vector<int64_t> seg_numel;
  std::vector<int32_t> seg_dtype;
  int64_t num_items = 0;
  int64_t bytes_per_step = 0;
  bool ptrs_bound = false;

  void* arena = nullptr;
  Item* d_items = nullptr;
  int64_t* d_unit_item_off = nullptr;
  const char** d_seg_base = nullptr;
  int32_t* d_seg_dtype = nullptr;
  uint8_t* d_rec = nullptr;
  float* d_partial = nullptr;
  double* d_A = nullptr;
  double* d_Q = nullptr;
  int32_t* d_lock = nullptr;
  double* d_norm = nullptr;
  double* d_gnmr = nullptr;
  double* d_dgnmr = nullptr;
  double* d_risk = nullptr;
  uint8_t* d_flags = nullptr;
  uint8_t* d_mask = nullptr;
  uint64_t* d_keys = nullptr;
  int32_t* d_counters = nullptr;
  int32_t* d_cand_list = nullptr;
  double* d_gsum = nullptr;
  gnmr_stats* d_stats = nullptr;
  int64_t* d_step = nullptr;   // steps completed (advanced by K3)

  // partial sums of squares made by a producer (gnmr_bind_partials)
  int64_t* d_ext_off = nullptr;  // [U+1]
  int64_t num_ext = -1;          // -1: none bound

  // pinned staging for segment-pointer uploads; `upload_done` guards reuse
  const void** h_ptr_stage = nullptr;
  hipEvent_t upload_done = nullptr;
  bool upload_pending = false;

  bool prof = false;
  std::vector<std::array<hipEvent_t, 4>> prof_ev;
  int64_t prof_steps = 0;
};

namespace {

// Checks a segment layout for U units: the CSR offsets, every segment's
// size and dtype, and the K1 item count (one workgroup per item, and a grid
// holds fewer than 2^32 lanes).
gnmr_status check_layout(const gnmr_segments* segs, int64_t U) {
  const int64_t S = segs->num_segments;
  if (S < 0 || S > INT32_MAX) return fail(GNMR_E_INVALID, "num_segments out of range");
  if (segs->unit_seg_off == nullptr) return fail(GNMR_E_INVALID, "unit_seg_off is NULL");
  if (S > 0 && (segs->seg_numel == nullptr || segs->seg_dtype == nullptr))
    return fail(GNMR_E_INVALID, "seg_numel or seg_dtype is NULL");
  if (segs->unit_seg_off[0] != 0 || segs->unit_seg_off[U] != S)
    return fail(GNMR_E_INVALID, "unit_seg_off must start at 0 and end at num_segments");
  for (int64_t b = 0; b < U; ++b)
    if (segs->unit_seg_off[b + 1] < segs->unit_seg_off[b])
      return fail(GNMR_E_INVALID, "unit_seg_off must be non-decreasing");
  const int64_t max_items = int64_t(UINT32_MAX) / gnmr::kK1Block;
  int64_t num_items = 0;
  for (int64_t s = 0; s < S; ++s) {
    const int64_t n = segs->seg_numel[s];
    if (n < 0) return fail(GNMR_E_INVALID, "negative seg_numel");
    if (segs->seg_dtype[s] != GNMR_F32 && segs->seg_dtype[s] != GNMR_BF16)
      return fail(GNMR_E_INVALID, "unknown seg_dtype " + std::to_string(segs->seg_dtype[s]));
    const int64_t per = gnmr::kItemBytes / (segs->seg_dtype[s] == GNMR_BF16 ? 2 : 4);
    if (n > (int64_t(1) << 50)) return fail(GNMR_E_INVALID, "seg_numel above 2^50");
    num_items += (n + per - 1) / per;  // at most 2^37 more: no overflow before the test
    if (num_items > max_items)
      return fail(GNMR_E_INVALID, "too many work items for one launch: more than " +
                                      std::to_string(max_items) +
                                      " (each segment takes one item per started 64 KiB)");
  }
  return GNMR_OK;
}

// The K1 work list of a checked layout: each segment cut into items of
// kItemBytes, in unit order; unit b owns items [unit_item_off[b],
// unit_item_off[b+1]).  Returns the gradient bytes of one pass.
int64_t build_work_list(const gnmr_segments* segs, int64_t U, std::vector<Item>* items,
                        std::vector<int64_t>* unit_item_off) {
  int64_t bytes = 0;
  items->clear();
  unit_item_off->assign(size_t(U) + 1, 0);
  for (int64_t b = 0; b < U; ++b) {
    for (int64_t s = segs->unit_seg_off[b]; s < segs->unit_seg_off[b + 1]; ++s) {
      const int64_t n = segs->seg_numel[s];
      const int64_t esz = segs->seg_dtype[s] == GNMR_BF16 ? 2 : 4;
      const int64_t per = gnmr::kItemBytes / esz;
      bytes += n * esz;
      for (int64_t e0 = 0; e0 < n; e0 += per)
        items->push_back(Item{e0, int32_t(s), int32_t(std::min(per, n - e0))});
    }
    (*unit_item_off)[size_t(b) + 1] = int64_t(items->size());
  }
  return bytes;
}

gnmr_status check_thresholds(double alpha, double beta) {
  if (!(alpha > 0.0) || !(beta > 0.0) || !isfinite(alpha) || !isfinite(beta))
    return fail(GNMR_E_INVALID, "alpha_t and beta_t must be finite and > 0");
  return GNMR_OK;
}

gnmr_status check_seg_ptrs(int64_t S, const int64_t* numel, const int32_t* dtype,
                           const void* const* ptrs) {
  for (int64_t s = 0; s < S; ++s) {
    if (numel[s] == 0) continue;
    const uintptr_t p = reinterpret_cast<uintptr_t>(ptrs[s]);
    const uintptr_t esz = dtype[s] == GNMR_BF16 ? 2 : 4;
    if (p == 0) return fail(GNMR_E_INVALID, "segment " + std::to_string(s) + ": NULL pointer");
    if (p % esz != 0)
      return fail(GNMR_E_INVALID,
                  "segment " + std::to_string(s) + ": pointer not aligned to its element size");
  }
  return GNMR_OK;
}

gnmr_status check_ptrs(const gnmr_ctx* c, const void* const* ptrs) {
  return check_seg_ptrs(c->S, c->seg_numel.data(), c->seg_dtype.data(), ptrs);
}

// Copies this step's segment pointers to the device table on `st`.
gnmr_status bind_ptrs(gnmr_ctx* c, const void* const* ptrs, hipStream_t st) {
  if (ptrs == nullptr) {
    if (!c->ptrs_bound && c->num_items > 0)
      return fail(GNMR_E_INVALID, "no segment pointers bound: pass seg_ptr");
    return GNMR_OK;
  }
  gnmr_status r = check_ptrs(c, ptrs);
  if (r != GNMR_OK) return r;
  if (c->S == 0) return GNMR_OK;
  if (c->upload_pending) {
    GNMR_HIP(hipEventSynchronize(c->upload_done));
    c->upload_pending = false;
  }
  memcpy(c->h_ptr_stage, ptrs, size_t(c->S) * sizeof(void*));
  GNMR_HIP(hipMemcpyAsync(c->d_seg_base, c->h_ptr_stage, size_t(c->S) * sizeof(void*),
                          hipMemcpyHostToDevice, st));
  GNMR_HIP(hipEventRecord(c->upload_done, st));
  c->upload_pending = true;
  c->ptrs_bound = true;
  return GNMR_OK;
}

gnmr_status record(gnmr_ctx* c, int which, hipStream_t st) {
  if (!c->prof || c->prof_steps >= kProfileCapacity) return GNMR_OK;
  if (size_t(c->prof_steps) >= c->prof_ev.size()) {
    std::array<hipEvent_t, 4> ev{};
    for (auto& e : ev) GNMR_HIP(hipEventCreate(&e));
    c->prof_ev.push_back(ev);
  }
  GNMR_HIP(hipEventRecord(c->prof_ev[size_t(c->prof_steps)][which], st));
  return GNMR_OK;
}

// K2 + K3 for step t+1 over the partial sums `partial` ([num_parts], unit b
// owning [off[b], off[b+1])), or over the norms ext_norm when it is non-null.
gnmr_status update_and_select(gnmr_ctx* c, const double* ext_norm, const float* partial,
                              const int64_t* off, int64_t num_parts, double alpha, double beta,
                              hipStream_t st) {
  gnmr::UpdateArgs u{};
  u.num_units = c->U;
  u.window = c->window;
  u.admitted = c->budget_mode == GNMR_BUDGET_ADMITTED ? 1 : 0;
  u.static_set = c->budget_mode == GNMR_BUDGET_STATIC ? 1 : 0;
  u.warmup = c->warmup_steps;
  u.step = c->d_step;
  u.gsum = c->d_gsum;
  u.eps = c->eps;
  u.alpha = alpha;
  u.beta = beta;
  u.unit_item_off = off;
  u.partial = partial;
  u.ext_norm = ext_norm;
  u.A = c->d_A;
  u.Q = c->d_Q;
  u.norm = c->d_norm;
  u.gnmr = c->d_gnmr;
  u.dgnmr = c->d_dgnmr;
  u.risk = c->d_risk;
  u.rec = c->d_rec;
  u.lock = c->d_lock;
  u.keys = c->d_keys;
  u.flags = c->d_flags;
  u.mask = c->d_mask;
  u.counters = c->d_counters;
  u.cand_list = c->d_cand_list;
  u.list_cap = gnmr::cand_list_cap(c->U);
  gnmr::SelectArgs s{};
  s.num_units = c->U;
  s.max_o = c->max_o;
  s.lock_len = u.static_set ? 0 : c->lock_len;   // the static baseline uses no locks
  s.warmup = c->warmup_steps;
  s.step = c->d_step;
  s.flags = c->d_flags;
  s.keys = c->d_keys;
  s.counters = c->d_counters;
  s.cand_list = c->d_cand_list;
  s.num_sets = gnmr::kCounterSets;
  s.list_cap = u.list_cap;
  s.lock = c->d_lock;
  s.mask = c->d_mask;
  s.stats = c->d_stats;
  gnmr_status r = GNMR_OK;
  if (gnmr::single_launch_update_select(u, num_parts)) {
    // small workload: K2 + K3 in one launch (timed as the update; select 0)
    GNMR_HIP(gnmr::launch_update_select(u, s, st));
    r = record(c, 2, st);
    if (r == GNMR_OK) r = record(c, 3, st);
    if (r != GNMR_OK) return r;
  } else {
    GNMR_HIP(gnmr::launch_update(u, num_parts, st));
    r = record(c, 2, st);
    if (r != GNMR_OK) return r;
    GNMR_HIP(gnmr::launch_select(s, st));
    r = record(c, 3, st);
    if (r != GNMR_OK) return r;
  }
  if (c->prof && c->prof_steps < kProfileCapacity) ++c->prof_steps;
  return GNMR_OK;
}

void release(gnmr_ctx* c) {
  if (c == nullptr) return;
  if (c->upload_done) (void)hipEventSynchronize(c->upload_done);
  for (auto& ev : c->prof_ev)
    for (auto e : ev)
      if (e) (void)hipEventDestroy(e);
  if (c->upload_done) (void)hipEventDestroy(c->upload_done);
  if (c->h_ptr_stage) (void)hipHostFree(c->h_ptr_stage);
  if (c->d_ext_off) {
    (void)hipDeviceSynchronize();
    (void)hipFree(c->d_ext_off);
  }
  if (c->arena) {
    (void)hipDeviceSynchronize();
    (void)hipFree(c->arena);
  }
  delete c;
}

}  // namespace

extern "C" {

const char* gnmr_last_error(void) { return g_last_error.c_str(); }

gnmr_status gnmr_init(gnmr_ctx** out, const gnmr_config* cfg, const gnmr_segments* segs,
                      void* stream) {
  if (out == nullptr) return fail(GNMR_E_INVALID, "out is NULL");
  *out = nullptr;
  if (cfg == nullptr || segs == nullptr) return fail(GNMR_E_INVALID, "cfg or segs is NULL");
  if (cfg->num_units < 1) return fail(GNMR_E_INVALID, "num_units must be >= 1");
  if (cfg->window < 1) return fail(GNMR_E_INVALID, "window must be >= 1");
  if (cfg->max_o < 0) return fail(GNMR_E_INVALID, "max_o must be >= 0");
  if (cfg->lock_len < 0) return fail(GNMR_E_INVALID, "lock_len must be >= 0");
  if (!(cfg->eps >= 0.0) || !isfinite(cfg->eps))
    return fail(GNMR_E_INVALID, "eps must be finite and >= 0");
  if (cfg->budget_mode != GNMR_BUDGET_ACTIVE && cfg->budget_mode != GNMR_BUDGET_ADMITTED &&
      cfg->budget_mode != GNMR_BUDGET_STATIC)
    return fail(GNMR_E_INVALID, "unknown budget_mode " + std::to_string(cfg->budget_mode));
  if (cfg->warmup_steps < 0) return fail(GNMR_E_INVALID, "warmup_steps must be >= 0");
  if (cfg->budget_mode == GNMR_BUDGET_STATIC && cfg->warmup_steps < 1)
    return fail(GNMR_E_INVALID, "the static baseline needs warmup_steps >= 1");
  const int64_t U = cfg->num_units, S = segs->num_segments;
  gnmr_status lr = check_layout(segs, U);
  if (lr != GNMR_OK) return lr;

  // K2 workgroups of 1, 4 or 256 units fill counter set w % kCounterSets:
  // each set's share of the candidate list must fit its capacity
  for (const int64_t per_wg : {int64_t(1), int64_t(4), int64_t(256)}) {
    const int64_t wgs = (U + per_wg - 1) / per_wg;
    if ((wgs + gnmr::kCounterSets - 1) / gnmr::kCounterSets * per_wg > gnmr::cand_list_cap(U))
      return fail(GNMR_E_INVALID, "candidate list layout does not fit (internal)");
  }

  gnmr_ctx* c = new (std::nothrow) gnmr_ctx;
  if (c == nullptr) return fail(GNMR_E_NOMEM, "host allocation failed");
  c->U = cfg->num_units;
  c->window = cfg->window;
  c->max_o = cfg->max_o;
  c->lock_len = cfg->lock_len;
  c->budget_mode = cfg->budget_mode;
  c->warmup_steps = cfg->warmup_steps;
  c->eps = cfg->eps;
  c->S = S;
  c->seg_numel.assign(segs->seg_numel, segs->seg_numel + S);
  c->seg_dtype.assign(segs->seg_dtype, segs->seg_dtype + S);
  if (segs->seg_ptr != nullptr) {
    gnmr_status r = check_ptrs(c, segs->seg_ptr);
    if (r != GNMR_OK) {
      delete c;
      return r;
    }
  }

  std::vector<Item> items;
  std::vector<int64_t> unit_item_off;
  c->bytes_per_step = build_work_list(segs, U, &items, &unit_item_off);
  c->num_items = int64_t(items.size());

  // One device arena for all state.
  const size_t a = 256;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + std::max<size_t>(bytes, 1), a);
    return o;
  };
  const size_t o_items = take(items.size() * sizeof(Item));
  const size_t o_uoff = take((size_t(U) + 1) * sizeof(int64_t));
  const size_t o_base = take(size_t(S) * sizeof(void*));
  const size_t o_dt = take(size_t(S) * sizeof(int32_t));
  const size_t o_rec = take(size_t(U));
  const size_t o_part = take(items.size() * sizeof(float));
  const size_t o_A = take(size_t(U) * sizeof(double));
  const size_t o_Q = take(size_t(U) * size_t(cfg->window) * sizeof(double));
  const size_t o_lock = take(size_t(U) * sizeof(int32_t));
  const size_t o_norm = take(size_t(U) * sizeof(double));
  const size_t o_g = take(size_t(U) * sizeof(double));
  const size_t o_d = take(size_t(U) * sizeof(double));
  const size_t o_r = take(size_t(U) * sizeof(double));
  const size_t o_fl = take(size_t(U));
  const size_t o_mask = take(size_t(U));
  const size_t o_keys = take(size_t(U) * sizeof(uint64_t));
  const size_t o_cnt = take(size_t(gnmr::kCounterSets) * gnmr::kNumCounters * sizeof(int32_t));
  const size_t o_list =
      take(size_t(gnmr::kCounterSets) * size_t(gnmr::cand_list_cap(U)) * sizeof(int32_t));
  const size_t o_gsum = take(size_t(U) * sizeof(double));
  const size_t o_st = take(sizeof(gnmr_stats));
  const size_t o_step = take(sizeof(int64_t));
  const size_t total = off;

  hipStream_t st = static_cast<hipStream_t>(stream);
  auto bail = [&](gnmr_status s, const std::string& m) {
    release(c);
    return fail(s, m);
  };
  if (hipGetDevice(&c->device) != hipSuccess) return bail(GNMR_E_HIP, "hipGetDevice failed");
  if (hipMalloc(&c->arena, total) != hipSuccess) {
    c->arena = nullptr;
    return bail(GNMR_E_NOMEM, "hipMalloc of " + std::to_string(total) + " bytes failed");
  }
  char* base = static_cast<char*>(c->arena);
  c->d_items = reinterpret_cast<Item*>(base + o_items);
  c->d_unit_item_off = reinterpret_cast<int64_t*>(base + o_uoff);
  c->d_seg_base = reinterpret_cast<const char**>(base + o_base);
  c->d_seg_dtype = reinterpret_cast<int32_t*>(base + o_dt);
  c->d_rec = reinterpret_cast<uint8_t*>(base + o_rec);
  c->d_partial = reinterpret_cast<float*>(base + o_part);
  c->d_A = reinterpret_cast<double*>(base + o_A);
  c->d_Q = reinterpret_cast<double*>(base + o_Q);
  c->d_lock = reinterpret_cast<int32_t*>(base + o_lock);
  c->d_norm = reinterpret_cast<double*>(base + o_norm);
  c->d_gnmr = reinterpret_cast<double*>(base + o_g);
  c->d_dgnmr = reinterpret_cast<double*>(base + o_d);
  c->d_risk = reinterpret_cast<double*>(base + o_r);
  c->d_flags = reinterpret_cast<uint8_t*>(base + o_fl);
  c->d_mask = reinterpret_cast<uint8_t*>(base + o_mask);
  c->d_keys = reinterpret_cast<uint64_t*>(base + o_keys);
  c->d_counters = reinterpret_cast<int32_t*>(base + o_cnt);
  c->d_cand_list = reinterpret_cast<int32_t*>(base + o_list);
  c->d_gsum = reinterpret_cast<double*>(base + o_gsum);
  c->d_stats = reinterpret_cast<gnmr_stats*>(base + o_st);
  c->d_step = reinterpret_cast<int64_t*>(base + o_step);

  if (hipHostMalloc(reinterpret_cast<void**>(&c->h_ptr_stage),
                    std::max<size_t>(size_t(S), 1) * sizeof(void*), hipHostMallocDefault) !=
      hipSuccess) {
    c->h_ptr_stage = nullptr;
    return bail(GNMR_E_NOMEM, "hipHostMalloc of the pointer staging buffer failed");
  }
  if (hipEventCreateWithFlags(&c->upload_done, hipEventDisableTiming) != hipSuccess) {
    c->upload_done = nullptr;
    return bail(GNMR_E_HIP, "hipEventCreate failed");
  }

  std::vector<uint8_t> rec(size_t(U), 1);
  if (cfg->recoverable != nullptr)
    for (int64_t b = 0; b < U; ++b) rec[size_t(b)] = cfg->recoverable[b] ? 1 : 0;

  hipError_t e = hipSuccess;
  if (!items.empty())
    e = hipMemcpyAsync(c->d_items, items.data(), items.size() * sizeof(Item),
                       hipMemcpyHostToDevice, st);
  if (e == hipSuccess)
    e = hipMemcpyAsync(c->d_unit_item_off, unit_item_off.data(),
                       unit_item_off.size() * sizeof(int64_t), hipMemcpyHostToDevice, st);
  if (e == hipSuccess && S > 0)
    e = hipMemcpyAsync(c->d_seg_dtype, c->seg_dtype.data(), size_t(S) * sizeof(int32_t),
                       hipMemcpyHostToDevice, st);
  if (e == hipSuccess)
    e = hipMemcpyAsync(c->d_rec, rec.data(), rec.size(), hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = hipMemsetAsync(c->d_A, 0, size_t(U) * sizeof(double), st);
  if (e == hipSuccess)
    e = hipMemsetAsync(c->d_Q, 0, size_t(U) * size_t(c->window) * sizeof(double), st);
  if (e == hipSuccess) e = hipMemsetAsync(c->d_lock, 0, size_t(U) * sizeof(int32_t), st);
  if (e == hipSuccess) e = hipMemsetAsync(c->d_mask, 0, size_t(U), st);
  if (e == hipSuccess) e = hipMemsetAsync(c->d_gsum, 0, size_t(U) * sizeof(double), st);
  if (e == hipSuccess) e = hipMemsetAsync(c->d_stats, 0, sizeof(gnmr_stats), st);
  if (e == hipSuccess) e = hipMemsetAsync(c->d_step, 0, sizeof(int64_t), st);
  if (e == hipSuccess)
    e = hipMemsetAsync(c->d_counters, 0,
                       size_t(gnmr::kCounterSets) * gnmr::kNumCounters * sizeof(int32_t), st);
  if (e == hipSuccess && S > 0)
    e = hipMemsetAsync(c->d_seg_base, 0, size_t(S) * sizeof(void*), st);
  // wait for what was enqueued also on failure: the uploads read host vectors
  // of this call and write the arena that bail() frees
  const hipError_t es = hipStreamSynchronize(st);
  if (e == hipSuccess) e = es;
  if (e != hipSuccess) return bail(GNMR_E_HIP, std::string("init upload: ") + hipGetErrorString(e));

  if (segs->seg_ptr != nullptr) {
    gnmr_status r = bind_ptrs(c, segs->seg_ptr, st);
    if (r == GNMR_OK && hipStreamSynchronize(st) != hipSuccess)
      r = fail(GNMR_E_HIP, "init pointer upload failed");
    if (r != GNMR_OK) {
      std::string m = g_last_error;
      return bail(r, m);
    }
  }
  *out = c;
  return GNMR_OK;
}

gnmr_status gnmr_destroy(gnmr_ctx* ctx) {
  if (ctx == nullptr) return GNMR_OK;
  DeviceGuard g(ctx->device);
  release(ctx);
  return GNMR_OK;
}

gnmr_status gnmr_step(gnmr_ctx* ctx, double alpha_t, double beta_t, const void* const* seg_ptr,
                      void* stream) {
  if (ctx == nullptr) return fail(GNMR_E_INVALID, "ctx is NULL");
  gnmr_status r = check_thresholds(alpha_t, beta_t);
  if (r != GNMR_OK) return r;
  DeviceGuard g(ctx->device);
  if (!g.ok) return fail(GNMR_E_HIP, "cannot select the context's device");
  hipStream_t st = static_cast<hipStream_t>(stream);
  r = bind_ptrs(ctx, seg_ptr, st);
  if (r != GNMR_OK) return r;
  r = record(ctx, 0, st);
  if (r != GNMR_OK) return r;
  GNMR_HIP(gnmr::launch_sumsq(ctx->d_items, ctx->num_items, ctx->d_seg_base, ctx->d_seg_dtype,
                              ctx->d_partial, st));
  r = record(ctx, 1, st);
  if (r != GNMR_OK) return r;
  return update_and_select(ctx, nullptr, ctx->d_partial, ctx->d_unit_item_off, ctx->num_items,
                           alpha_t, beta_t, st);
}

gnmr_status gnmr_step_from_norms(gnmr_ctx* ctx, const double* d_norm, double alpha_t,
                                 double beta_t, void* stream) {
  if (ctx == nullptr) return fail(GNMR_E_INVALID, "ctx is NULL");
  if (d_norm == nullptr) return fail(GNMR_E_INVALID, "d_norm is NULL");
  gnmr_status r = check_thresholds(alpha_t, beta_t);
  if (r != GNMR_OK) return r;
  DeviceGuard g(ctx->device);
  if (!g.ok) return fail(GNMR_E_HIP, "cannot select the context's device");
  hipStream_t st = static_cast<hipStream_t>(stream);
  r = record(ctx, 0, st);
  if (r == GNMR_OK) r = record(ctx, 1, st);
  if (r != GNMR_OK) return r;
  return update_and_select(ctx, d_norm, ctx->d_partial, ctx->d_unit_item_off, ctx->num_items,
                           alpha_t, beta_t, st);
}

gnmr_status gnmr_bind_partials(gnmr_ctx* ctx, int64_t num_partials,
                               const int64_t* unit_part_off) {
  if (ctx == nullptr) return fail(GNMR_E_INVALID, "ctx is NULL");
  if (unit_part_off == nullptr) return fail(GNMR_E_INVALID, "unit_part_off is NULL");
  if (num_partials < 0) return fail(GNMR_E_INVALID, "num_partials must be >= 0");
  if (unit_part_off[0] != 0 || unit_part_off[ctx->U] != num_partials)
    return fail(GNMR_E_INVALID, "unit_part_off must start at 0 and end at num_partials");
  for (int32_t b = 0; b < ctx->U; ++b)
    if (unit_part_off[b + 1] < unit_part_off[b])
      return fail(GNMR_E_INVALID, "unit_part_off must be non-decreasing");
  DeviceGuard g(ctx->device);
  if (!g.ok) return fail(GNMR_E_HIP, "cannot select the context's device");
  const size_t bytes = size_t(ctx->U + 1) * sizeof(int64_t);
  if (ctx->d_ext_off == nullptr) GNMR_HIP(hipMalloc(&ctx->d_ext_off, bytes));
  GNMR_HIP(hipDeviceSynchronize());
  GNMR_HIP(hipMemcpy(ctx->d_ext_off, unit_part_off, bytes, hipMemcpyHostToDevice));
  ctx->num_ext = num_partials;
  return GNMR_OK;
}

gnmr_status gnmr_step_from_partials(gnmr_ctx* ctx, const float* d_partial, double alpha_t,
                                    double beta_t, void* stream) {
  if (ctx == nullptr) return fail(GNMR_E_INVALID, "ctx is NULL");
  if (ctx->num_ext < 0) return fail(GNMR_E_STATE, "no partial layout bound (gnmr_bind_partials)");
  if (d_partial == nullptr && ctx->num_ext > 0) return fail(GNMR_E_INVALID, "d_partial is NULL");
  gnmr_status r = check_thresholds(alpha_t, beta_t);
  if (r != GNMR_OK) return r;
  DeviceGuard g(ctx->device);
  if (!g.ok) return fail(GNMR_E_HIP, "cannot select the context's device");
  hipStream_t st = static_cast<hipStream_t>(stream);
  r = record(ctx, 0, st);
  if (r == GNMR_OK) r = record(ctx, 1, st);
  if (r != GNMR_OK) return r;
  return update_and_select(ctx, nullptr, d_partial, ctx->d_ext_off, ctx->num_ext, alpha_t, beta_t,
                           st);
}

int64_t gnmr_wgrad_num_tiles(int32_t out_features, int32_t in_features) {
  if (out_features <= 0 || in_features <= 0) return 0;
  return gnmr::wgrad_tiles(out_features, in_features);
}

constexpr int64_t kWgMaxTiles = int64_t(UINT32_MAX) / gnmr::kWgThreads;

gnmr_status gnmr_wgrad_sumsq_batched(const gnmr_wgrad_problem* problems, int32_t num_problems,
                                     float* tile_sumsq, void* stream) {
  if (num_problems < 0 || (num_problems > 0 && problems == nullptr))
    return fail(GNMR_E_INVALID, "problems must hold num_problems >= 0 entries");
  if (num_problems > 0 && tile_sumsq == nullptr)
    return fail(GNMR_E_INVALID, "tile_sumsq must be a device pointer");
  for (int32_t i = 0; i < num_problems; ++i) {
    const gnmr_wgrad_problem& q = problems[i];
    if (q.out_features <= 0 || q.in_features <= 0 || q.tokens < 0)
      return fail(GNMR_E_INVALID, "out_features and in_features must be > 0, tokens >= 0");
    if (q.out_features % 8 != 0 || q.in_features % 8 != 0)
      return fail(GNMR_E_INVALID, "out_features and in_features must be multiples of 8");
    // K5 addresses one K step of an operand (64 rows) with 32-bit byte offsets
    if (q.out_features >= (1 << 24) || q.in_features >= (1 << 24))
      return fail(GNMR_E_INVALID, "out_features and in_features must be < 2^24");
    if (q.dw == nullptr || (q.tokens > 0 && (q.dy == nullptr || q.x == nullptr)))
      return fail(GNMR_E_INVALID, "dy, x and dw must be device pointers");
    if ((reinterpret_cast<uintptr_t>(q.dy) | reinterpret_cast<uintptr_t>(q.x) |
         reinterpret_cast<uintptr_t>(q.dw)) % 16 != 0)
      return fail(GNMR_E_INVALID, "dy, x and dw must be 16-byte aligned");
    // one workgroup of kWgThreads lanes per tile; a grid holds < 2^32 lanes
    if (gnmr::wgrad_tiles(q.out_features, q.in_features) > kWgMaxTiles)
      return fail(GNMR_E_INVALID, "too many output tiles for one launch");
    if (q.accumulate != 0 && q.accumulate != 1)
      return fail(GNMR_E_INVALID, "accumulate must be 0 or 1");
    if (q.reserved != 0) return fail(GNMR_E_INVALID, "reserved must be 0");
  }
  // No write may race another access: each dw and the tile sums are disjoint
  // from one another and from every operand of the batch.
  {
    std::vector<Span> w, r;
    int64_t tiles = 0;
    for (int32_t i = 0; i < num_problems; ++i) {
      const gnmr_wgrad_problem& q = problems[i];
      const Span dw = span_of(q.dw, int64_t(q.out_features) * q.in_features * 2, i);
      const Span dy = span_of(q.dy, q.tokens * q.out_features * 2, i);
      const Span x = span_of(q.x, q.tokens * q.in_features * 2, i);
      if (intersect(dw, dy) || intersect(dw, x))
        return fail(GNMR_E_INVALID, "problem " + std::to_string(i) + ": dw overlaps dy or x");
      w.push_back(dw);
      r.push_back(dy);
      r.push_back(x);
      tiles += gnmr::wgrad_tiles(q.out_features, q.in_features);
    }
    w.push_back(span_of(tile_sumsq, tiles * int64_t(sizeof(float)), -2));
    if (find_overlap(w, r) != -1)
      return fail(GNMR_E_INVALID,
                  "a problem's dw or tile_sumsq overlaps another output or another problem's "
                  "operands");
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  int64_t base = 0;  // first partial of the current launch
  for (int32_t i = 0; i < num_problems;) {
    gnmr::WgBatch b{};
    int64_t tiles = 0;
    while (i < num_problems && b.num < gnmr::kWgMaxBatch) {
      const gnmr_wgrad_problem& q = problems[i];
      const int64_t t = gnmr::wgrad_tiles(q.out_features, q.in_features);
      if (b.num > 0 && tiles + t > kWgMaxTiles) break;
      gnmr::WgProblem& P = b.p[b.num++];
      P.dy = static_cast<const uint16_t*>(q.dy);
      P.x = static_cast<const uint16_t*>(q.x);
      P.dw = static_cast<uint16_t*>(q.dw);
      P.tile_ss = tile_sumsq + base + tiles;
      P.K = q.tokens;
      P.M = q.out_features;
      P.N = q.in_features;
      P.tiles_m = (q.out_features + gnmr::kWgBM - 1) / gnmr::kWgBM;
      P.tiles_n = (q.in_features + gnmr::kWgBN - 1) / gnmr::kWgBN;
      P.tile_begin = int32_t(tiles);
      P.accumulate = q.accumulate;
      tiles += t;
      ++i;
    }
    b.total_tiles = int32_t(tiles);
    GNMR_HIP(gnmr::launch_wgrad(b, st));
    base += tiles;
  }
  return GNMR_OK;
}

gnmr_status gnmr_wgrad_sumsq(const void* dy, const void* x, void* dw, int64_t tokens,
                             int32_t out_features, int32_t in_features, float* tile_sumsq,
                             void* stream) {
  if (tile_sumsq == nullptr) return fail(GNMR_E_INVALID, "tile_sumsq must be a device pointer");
  const gnmr_wgrad_problem q{dy, x, dw, tokens, out_features, in_features, 0, 0};
  return gnmr_wgrad_sumsq_batched(&q, 1, tile_sumsq, stream);
}

gnmr_status gnmr_sumsq(gnmr_ctx* ctx, const void* const* seg_ptr, double* d_sumsq,
                       void* stream) {
  if (ctx == nullptr) return fail(GNMR_E_INVALID, "ctx is NULL");
  if (d_sumsq == nullptr) return fail(GNMR_E_INVALID, "d_sumsq is NULL");
  DeviceGuard g(ctx->device);
  if (!g.ok) return fail(GNMR_E_HIP, "cannot select the context's device");
  hipStream_t st = static_cast<hipStream_t>(stream);
  gnmr_status r = bind_ptrs(ctx, seg_ptr, st);
  if (r != GNMR_OK) return r;
  GNMR_HIP(gnmr::launch_sumsq(ctx->d_items, ctx->num_items, ctx->d_seg_base, ctx->d_seg_dtype,
                              ctx->d_partial, st));
  GNMR_HIP(gnmr::launch_unit_sumsq(ctx->d_unit_item_off, ctx->d_partial, ctx->num_items,
                                   ctx->U, d_sumsq, st));
  return GNMR_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// The gradient pass without allocation: the work list and the item partials
// live in `scratch`, a fixed device array of the library (each device holds
// its own copy for the life of the process).  Host code reaches it only
// through the address hipGetSymbolAddress gives on that device: the array's
// name is not a device address in host code.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = GNMR_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on the current device, looked up on the
// first call there (with that device current) and kept.
gnmr_status scratch_address(void** out) {
  int dev = -1;
  GNMR_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(GNMR_E_HIP, "device index " + std::to_string(dev) + " out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    GNMR_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (p == nullptr) return fail(GNMR_E_HIP, "hipGetSymbolAddress gave no address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return GNMR_OK;
}

}  // namespace

extern "C" {

gnmr_status gnmr_sumsq_noalloc(int32_t num_units, const gnmr_segments* segs, double* d_sumsq,
                               void* stream) {
  if (num_units < 1) return fail(GNMR_E_INVALID, "num_units must be >= 1");
  if (segs == nullptr) return fail(GNMR_E_INVALID, "segs is NULL");
  if (d_sumsq == nullptr) return fail(GNMR_E_INVALID, "d_sumsq is NULL");
  const int64_t U = num_units, S = segs->num_segments;
  gnmr_status r = check_layout(segs, U);
  if (r != GNMR_OK) return r;
  if (S > 0 && segs->seg_ptr == nullptr)
    return fail(GNMR_E_INVALID, "seg_ptr is NULL: this call binds no pointers beforehand");
  r = check_seg_ptrs(S, segs->seg_numel, segs->seg_dtype, segs->seg_ptr);
  if (r != GNMR_OK) return r;
  std::vector<Item> items;
  std::vector<int64_t> unit_item_off;
  build_work_list(segs, U, &items, &unit_item_off);
  const int64_t n_items = int64_t(items.size());
  // scratch layout: item table, unit offsets, segment bases and dtypes (one
  // upload), then the item partials
  const size_t o_items = 0;
  const size_t o_uoff = align_up(o_items + size_t(n_items) * sizeof(Item), 256);
  const size_t o_base = align_up(o_uoff + (size_t(U) + 1) * sizeof(int64_t), 256);
  const size_t o_dt = align_up(o_base + size_t(S) * sizeof(void*), 256);
  const size_t o_part = align_up(o_dt + size_t(S) * sizeof(int32_t), 256);
  const size_t total = o_part + size_t(n_items) * sizeof(float);
  if (total > kScratchBytes)
    return fail(GNMR_E_INVALID, "the layout needs " + std::to_string(total) +
                                    " bytes of scratch (work list and partials); the "
                                    "allocation-free pass holds " +
                                    std::to_string(kScratchBytes));
  void* sp = nullptr;
  r = scratch_address(&sp);
  if (r != GNMR_OK) return r;
  std::vector<unsigned char> blob(o_part, 0);
  memcpy(blob.data() + o_items, items.data(), size_t(n_items) * sizeof(Item));
  memcpy(blob.data() + o_uoff, unit_item_off.data(), (size_t(U) + 1) * sizeof(int64_t));
  if (S > 0) {
    memcpy(blob.data() + o_base, segs->seg_ptr, size_t(S) * sizeof(void*));
    memcpy(blob.data() + o_dt, segs->seg_dtype, size_t(S) * sizeof(int32_t));
  }
  char* base = static_cast<char*>(sp);
  hipStream_t st = static_cast<hipStream_t>(stream);
  // ordered after earlier work on `stream`, so a previous call's kernels have
  // read the old work list before it is replaced
  GNMR_HIP(hipMemcpyAsync(base, blob.data(), blob.size(), hipMemcpyHostToDevice, st));
  hipError_t e = gnmr::launch_sumsq(reinterpret_cast<const Item*>(base + o_items), n_items,
                                    reinterpret_cast<const char* const*>(base + o_base),
                                    reinterpret_cast<const int32_t*>(base + o_dt),
                                    reinterpret_cast<float*>(base + o_part), st);
  if (e == hipSuccess)
    e = gnmr::launch_unit_sumsq(reinterpret_cast<const int64_t*>(base + o_uoff),
                                reinterpret_cast<const float*>(base + o_part), n_items,
                                num_units, d_sumsq, st);
  // the host copy of the work list must outlive the upload, also when a
  // launch failed after it was enqueued
  const hipError_t es = hipStreamSynchronize(st);
  if (e != hipSuccess) return fail(GNMR_E_HIP, std::string("launch: ") + hipGetErrorString(e));
  if (es != hipSuccess)
    return fail(GNMR_E_HIP, std::string("hipStreamSynchronize: ") + hipGetErrorString(es));
  return GNMR_OK;
}

gnmr_status gnmr_query(gnmr_ctx* ctx, uint8_t* mask, int32_t* lock, double* norm, double* gnmr,
                       double* dgnmr, double* risk, gnmr_stats* stats, void* stream) {
  if (ctx == nullptr) return fail(GNMR_E_INVALID, "ctx is NULL");
  DeviceGuard g(ctx->device);
  if (!g.ok) return fail(GNMR_E_HIP, "cannot select the context's device");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const size_t U = size_t(ctx->U);
  auto d2h = [&](void* dst, const void* src, size_t bytes) -> hipError_t {
    if (dst == nullptr) return hipSuccess;
    return hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, st);
  };
  GNMR_HIP(d2h(mask, ctx->d_mask, U));
  GNMR_HIP(d2h(lock, ctx->d_lock, U * sizeof(int32_t)));
  GNMR_HIP(d2h(norm, ctx->d_norm, U * sizeof(double)));
  GNMR_HIP(d2h(gnmr, ctx->d_gnmr, U * sizeof(double)));
  GNMR_HIP(d2h(dgnmr, ctx->d_dgnmr, U * sizeof(double)));
  GNMR_HIP(d2h(risk, ctx->d_risk, U * sizeof(double)));
  gnmr_stats local;
  GNMR_HIP(d2h(&local, ctx->d_stats, sizeof(gnmr_stats)));
  GNMR_HIP(hipStreamSynchronize(st));
  if (local.t == 0) return fail(GNMR_E_STATE, "no step has been taken yet");
  if (stats) *stats = local;
  return GNMR_OK;
}

gnmr_status gnmr_device_outputs(gnmr_ctx* ctx, const uint8_t** mask, const int32_t** lock,
                                const double** norm, const double** gnmr, const double** dgnmr,
                                const double** risk, const gnmr_stats** stats) {
  if (ctx == nullptr) return fail(GNMR_E_INVALID, "ctx is NULL");
  if (mask) *mask = ctx->d_mask;
  if (lock) *lock = ctx->d_lock;
  if (norm) *norm = ctx->d_norm;
  if (gnmr) *gnmr = ctx->d_gnmr;
  if (dgnmr) *dgnmr = ctx->d_dgnmr;
  if (risk) *risk = ctx->d_risk;
  if (stats) *stats = ctx->d_stats;
  return GNMR_OK;
}

gnmr_status gnmr_state_size(const gnmr_ctx* ctx, size_t* bytes) {
  if (ctx == nullptr || bytes == nullptr) return fail(GNMR_E_INVALID, "NULL argument");
  const size_t U = size_t(ctx->U);
  *bytes = sizeof(StateHeader) + U * sizeof(double) * (1 + size_t(ctx->window)) +
           U * sizeof(int32_t) + U + U * sizeof(double);
  return GNMR_OK;
}

gnmr_status gnmr_get_state(gnmr_ctx* ctx, void* buf, size_t bytes, void* stream) {
  size_t need = 0;
  gnmr_status r = gnmr_state_size(ctx, &need);
  if (r != GNMR_OK) return r;
  if (buf == nullptr || bytes < need) return fail(GNMR_E_INVALID, "state buffer too small");
  DeviceGuard g(ctx->device);
  if (!g.ok) return fail(GNMR_E_HIP, "cannot select the context's device");
  hipStream_t st = static_cast<hipStream_t>(stream);
  int64_t t = 0;
  GNMR_HIP(hipMemcpyAsync(&t, ctx->d_step, sizeof(int64_t), hipMemcpyDeviceToHost, st));
  GNMR_HIP(hipStreamSynchronize(st));
  StateHeader h{kStateMagic, kStateVersion, ctx->U,        ctx->window,      t,
                ctx->max_o,  ctx->lock_len,  ctx->eps, ctx->budget_mode, ctx->warmup_steps};
  char* p = static_cast<char*>(buf);
  memcpy(p, &h, sizeof h);
  p += sizeof h;
  const size_t U = size_t(ctx->U);
  GNMR_HIP(hipMemcpyAsync(p, ctx->d_A, U * sizeof(double), hipMemcpyDeviceToHost, st));
  p += U * sizeof(double);
  GNMR_HIP(hipMemcpyAsync(p, ctx->d_Q, U * size_t(ctx->window) * sizeof(double),
                          hipMemcpyDeviceToHost, st));
  p += U * size_t(ctx->window) * sizeof(double);
  GNMR_HIP(hipMemcpyAsync(p, ctx->d_lock, U * sizeof(int32_t), hipMemcpyDeviceToHost, st));
  p += U * sizeof(int32_t);
  GNMR_HIP(hipMemcpyAsync(p, ctx->d_mask, U, hipMemcpyDeviceToHost, st));
  p += U;
  GNMR_HIP(hipMemcpyAsync(p, ctx->d_gsum, U * sizeof(double), hipMemcpyDeviceToHost, st));
  GNMR_HIP(hipStreamSynchronize(st));
  return GNMR_OK;
}

gnmr_status gnmr_set_state(gnmr_ctx* ctx, const void* buf, size_t bytes, void* stream) {
  size_t need = 0;
  gnmr_status r = gnmr_state_size(ctx, &need);
  if (r != GNMR_OK) return r;
  if (buf == nullptr || bytes != need) return fail(GNMR_E_INVALID, "state blob size mismatch");
  StateHeader h;
  memcpy(&h, buf, sizeof h);
  if (h.magic != kStateMagic || h.version != kStateVersion)
    return fail(GNMR_E_INVALID, "not a GNMR state blob of this version");
  if (h.num_units != ctx->U || h.window != ctx->window)
    return fail(GNMR_E_INVALID, "state blob is for a different num_units or window");
  // The blob's Lock values lie in [0, T_lock] and its queue, sums and A_{t-1}
  // follow one budget convention: a context with other settings would step on
  // from a state its own run could never reach.
  if (h.max_o != ctx->max_o || h.lock_len != ctx->lock_len ||
      h.eps != ctx->eps || h.budget_mode != ctx->budget_mode ||
      h.warmup_steps != ctx->warmup_steps)
    return fail(GNMR_E_INVALID,
                "state blob is for different max_o, lock_len, eps, budget_mode or warmup_steps");
  if (h.t < 0) return fail(GNMR_E_INVALID, "state blob has a negative step counter");
  DeviceGuard g(ctx->device);
  if (!g.ok) return fail(GNMR_E_HIP, "cannot select the context's device");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const char* p = static_cast<const char*>(buf) + sizeof h;
  const size_t U = size_t(ctx->U);
  GNMR_HIP(hipMemcpyAsync(ctx->d_A, p, U * sizeof(double), hipMemcpyHostToDevice, st));
  p += U * sizeof(double);
  GNMR_HIP(hipMemcpyAsync(ctx->d_Q, p, U * size_t(ctx->window) * sizeof(double),
                          hipMemcpyHostToDevice, st));
  p += U * size_t(ctx->window) * sizeof(double);
  GNMR_HIP(hipMemcpyAsync(ctx->d_lock, p, U * sizeof(int32_t), hipMemcpyHostToDevice, st));
  p += U * sizeof(int32_t);
  GNMR_HIP(hipMemcpyAsync(ctx->d_mask, p, U, hipMemcpyHostToDevice, st));
  p += U;
  GNMR_HIP(hipMemcpyAsync(ctx->d_gsum, p, U * sizeof(double), hipMemcpyHostToDevice, st));
  GNMR_HIP(hipMemcpyAsync(ctx->d_step, &h.t, sizeof(int64_t), hipMemcpyHostToDevice, st));
  // The per-step outputs are not part of the state: clear the counters (t = 0)
  // so that gnmr_query reports GNMR_E_STATE until the next step writes them.
  GNMR_HIP(hipMemsetAsync(ctx->d_stats, 0, sizeof(gnmr_stats), st));
  GNMR_HIP(hipStreamSynchronize(st));
  return GNMR_OK;
}

gnmr_status gnmr_set_profiling(gnmr_ctx* ctx, int enable) {
  if (ctx == nullptr) return fail(GNMR_E_INVALID, "ctx is NULL");
  ctx->prof = enable != 0;
  ctx->prof_steps = 0;
  return GNMR_OK;
}

gnmr_status gnmr_profile_read(gnmr_ctx* ctx, double* ms_sumsq, double* ms_update,
                              double* ms_select, int64_t* steps) {
  if (ctx == nullptr) return fail(GNMR_E_INVALID, "ctx is NULL");
  DeviceGuard g(ctx->device);
  double acc[3] = {0, 0, 0};
  for (int64_t i = 0; i < ctx->prof_steps; ++i) {
    auto& ev = ctx->prof_ev[size_t(i)];
    GNMR_HIP(hipEventSynchronize(ev[3]));
    for (int k = 0; k < 3; ++k) {
      float ms = 0.f;
      GNMR_HIP(hipEventElapsedTime(&ms, ev[k], ev[k + 1]));
      acc[k] += ms;
    }
  }
  if (ms_sumsq) *ms_sumsq = acc[0];
  if (ms_update) *ms_update = acc[1];
  if (ms_select) *ms_select = acc[2];
  if (steps) *steps = ctx->prof_steps;
  return GNMR_OK;
}

gnmr_status gnmr_info(const gnmr_ctx* ctx, int64_t* num_items, int64_t* item_bytes,
                      int64_t* bytes_per_step, int32_t* launches_per_step) {
  if (ctx == nullptr) return fail(GNMR_E_INVALID, "ctx is NULL");
  if (num_items) *num_items = ctx->num_items;
  if (item_bytes) *item_bytes = gnmr::kItemBytes;
  if (bytes_per_step) *bytes_per_step = ctx->bytes_per_step;
  if (launches_per_step) {
    gnmr::UpdateArgs u{};
    u.num_units = ctx->U;
    *launches_per_step = (ctx->num_items > 0 ? 1 : 0) +
                         (gnmr::single_launch_update_select(u, ctx->num_items) ? 1 : 2);
  }
  return GNMR_OK;
}

// ---------------------------------------------------------------------------
// recovery actuator
// ---------------------------------------------------------------------------

struct gnmr_actuator {
  int device = 0;
  int32_t num_units = 0;
  int64_t rows = 0;
  int64_t narrow_rows = 0;  // rows [0, narrow_rows) of the list take one wavefront each
  int64_t bytes = 0;
  void* arena = nullptr;
  gnmr::RowItem* d_items = nullptr;
  gnmr::ActSeg* d_segs = nullptr;
};

gnmr_status gnmr_actuator_create(gnmr_actuator** out, const gnmr_act_segment* segs,
                                 int64_t num_segments, int32_t num_units, void* stream) {
  if (out == nullptr) return fail(GNMR_E_INVALID, "out is NULL");
  *out = nullptr;
  if (num_segments < 0 || num_segments > INT32_MAX || (num_segments > 0 && segs == nullptr))
    return fail(GNMR_E_INVALID, "bad segment list");
  if (num_units < 1) return fail(GNMR_E_INVALID, "num_units must be >= 1");
  int64_t rows = 0, bytes = 0;
  for (int64_t k = 0; k < num_segments; ++k) {
    const gnmr_act_segment& g = segs[k];
    const std::string at = "activation segment " + std::to_string(k) + ": ";
    if (g.rows < 0) return fail(GNMR_E_INVALID, at + "negative rows");
    if (g.cols < 8 || g.cols > gnmr::kK4MaxCols || g.cols % 8 != 0)
      return fail(GNMR_E_INVALID, at + "cols must be a multiple of 8 in [8, 16384]");
    if (g.unit < 0 || g.unit >= num_units) return fail(GNMR_E_INVALID, at + "unit out of range");
    if (g.rows > 0) {
      if (g.in == nullptr || g.out == nullptr) return fail(GNMR_E_INVALID, at + "NULL pointer");
      if (reinterpret_cast<uintptr_t>(g.in) % 16 || reinterpret_cast<uintptr_t>(g.out) % 16)
        return fail(GNMR_E_INVALID, at + "pointers must be 16-byte aligned");
      if (g.rows > INT32_MAX) return fail(GNMR_E_INVALID, at + "too many rows");
    }
    rows += g.rows;
    bytes += g.rows * int64_t(g.cols) * 2;
  }
  if (rows > int64_t(UINT32_MAX)) return fail(GNMR_E_INVALID, "too many rows in total");
  {
    int64_t narrow_rows = 0;
    for (int64_t k = 0; k < num_segments; ++k)
      if (segs[k].cols <= gnmr::kK4WaveCols) narrow_rows += segs[k].rows;
    if (narrow_rows > 4 * gnmr::kK4MaxWorkgroups || rows - narrow_rows > gnmr::kK4MaxWorkgroups)
      return fail(GNMR_E_INVALID, "too many rows for one launch: at most " +
                                      std::to_string(4 * gnmr::kK4MaxWorkgroups) +
                                      " rows of up to 4096 features and " +
                                      std::to_string(gnmr::kK4MaxWorkgroups) + " longer rows");
  }
  // A segment writes in place or into memory that no segment reads, and no
  // two segments write the same bytes.
  {
    std::vector<Span> w, r;
    for (int64_t k = 0; k < num_segments; ++k) {
      const int64_t nb = segs[k].rows * int64_t(segs[k].cols) * 2;
      const Span in = span_of(segs[k].in, nb, k), out = span_of(segs[k].out, nb, k);
      if (in.lo != out.lo && intersect(in, out))
        return fail(GNMR_E_INVALID, "activation segment " + std::to_string(k) +
                                        ": out partly overlaps in (in place needs out == in)");
      w.push_back(out);
      r.push_back(in);
    }
    const int64_t k = find_overlap(w, r);
    if (k != -1)
      return fail(GNMR_E_INVALID, "activation segment " + std::to_string(k) +
                                      ": out overlaps another segment's input or output");
  }
  // Row list: the rows that one wavefront handles first, then the longer ones.
  std::vector<gnmr::RowItem> items;
  items.reserve(size_t(rows));
  std::vector<gnmr::ActSeg> dsegs(static_cast<size_t>(num_segments));
  for (int64_t k = 0; k < num_segments; ++k)
    dsegs[size_t(k)] = gnmr::ActSeg{static_cast<const char*>(segs[k].in),
                                    static_cast<char*>(segs[k].out), segs[k].cols, segs[k].unit};
  for (int pass = 0; pass < 2; ++pass)
    for (int64_t k = 0; k < num_segments; ++k)
      if ((segs[k].cols <= gnmr::kK4WaveCols) == (pass == 0))
        for (int64_t r = 0; r < segs[k].rows; ++r)
          items.push_back(gnmr::RowItem{int32_t(k), int32_t(r)});
  int64_t narrow = 0;
  for (int64_t k = 0; k < num_segments; ++k)
    if (segs[k].cols <= gnmr::kK4WaveCols) narrow += segs[k].rows;
  gnmr_actuator* a = new (std::nothrow) gnmr_actuator;
  if (a == nullptr) return fail(GNMR_E_NOMEM, "host allocation failed");
  a->num_units = num_units;
  a->rows = rows;
  a->narrow_rows = narrow;
  a->bytes = bytes;
  const size_t o_items = 0;
  const size_t o_segs = align_up(std::max<size_t>(items.size() * sizeof(gnmr::RowItem), 1), 256);
  const size_t total = o_segs + std::max<size_t>(dsegs.size() * sizeof(gnmr::ActSeg), 1);
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = hipGetDevice(&a->device);
  if (e == hipSuccess) e = hipMalloc(&a->arena, total);
  if (e != hipSuccess) {
    a->arena = nullptr;
    delete a;
    return fail(GNMR_E_NOMEM, "hipMalloc of the actuator tables failed");
  }
  a->d_items = reinterpret_cast<gnmr::RowItem*>(static_cast<char*>(a->arena) + o_items);
  a->d_segs = reinterpret_cast<gnmr::ActSeg*>(static_cast<char*>(a->arena) + o_segs);
  if (!items.empty())
    e = hipMemcpyAsync(a->d_items, items.data(), items.size() * sizeof(gnmr::RowItem),
                       hipMemcpyHostToDevice, st);
  if (e == hipSuccess && !dsegs.empty())
    e = hipMemcpyAsync(a->d_segs, dsegs.data(), dsegs.size() * sizeof(gnmr::ActSeg),
                       hipMemcpyHostToDevice, st);
  // wait for what was enqueued also on failure, before the arena is freed
  const hipError_t es = hipStreamSynchronize(st);
  if (e == hipSuccess) e = es;
  if (e != hipSuccess) {
    (void)hipFree(a->arena);
    delete a;
    return fail(GNMR_E_HIP, std::string("actuator upload: ") + hipGetErrorString(e));
  }
  *out = a;
  return GNMR_OK;
}

gnmr_status gnmr_actuate(gnmr_actuator* act, const uint8_t* d_mask, int32_t fmt_low,
                         int32_t fmt_recovery, void* stream) {
  if (act == nullptr || d_mask == nullptr) return fail(GNMR_E_INVALID, "NULL argument");
  if (fmt_low < GNMR_FMT_BF16 || fmt_low > GNMR_FMT_INT8 || fmt_recovery < GNMR_FMT_BF16 ||
      fmt_recovery > GNMR_FMT_INT8)
    return fail(GNMR_E_INVALID, "unknown format");
  DeviceGuard g(act->device);
  if (!g.ok) return fail(GNMR_E_HIP, "cannot select the actuator's device");
  GNMR_HIP(gnmr::launch_actuate(act->d_items, act->narrow_rows, act->rows, act->d_segs, d_mask,
                                fmt_low, fmt_recovery, static_cast<hipStream_t>(stream)));
  return GNMR_OK;
}

gnmr_status gnmr_actuate_matrix(const void* in, void* out, int64_t rows, int32_t cols,
                                const uint8_t* d_mask, int32_t unit, int32_t fmt_low,
                                int32_t fmt_recovery, void* stream) {
  if (rows < 0 || rows > INT32_MAX) return fail(GNMR_E_INVALID, "rows must be in [0, 2^31)");
  if (cols < 8 || cols > gnmr::kK4MaxCols || cols % 8 != 0)
    return fail(GNMR_E_INVALID, "cols must be a multiple of 8 in [8, 16384]");
  if (rows > (cols <= gnmr::kK4WaveCols ? 4 : 1) * gnmr::kK4MaxWorkgroups)
    return fail(GNMR_E_INVALID, "too many rows for one launch: at most " +
                                    std::to_string(4 * gnmr::kK4MaxWorkgroups) +
                                    " rows of up to 4096 features or " +
                                    std::to_string(gnmr::kK4MaxWorkgroups) + " longer rows");
  if (unit < 0) return fail(GNMR_E_INVALID, "unit must be >= 0");
  if (fmt_low < GNMR_FMT_BF16 || fmt_low > GNMR_FMT_INT8 || fmt_recovery < GNMR_FMT_BF16 ||
      fmt_recovery > GNMR_FMT_INT8)
    return fail(GNMR_E_INVALID, "unknown format");
  if (rows == 0) return GNMR_OK;
  if (in == nullptr || out == nullptr || d_mask == nullptr)
    return fail(GNMR_E_INVALID, "NULL argument");
  if (reinterpret_cast<uintptr_t>(in) % 16 || reinterpret_cast<uintptr_t>(out) % 16)
    return fail(GNMR_E_INVALID, "in and out must be 16-byte aligned");
  const int64_t nb = rows * int64_t(cols) * 2;
  const Span si = span_of(in, nb, 0), so = span_of(out, nb, 0);
  if (si.lo != so.lo && intersect(si, so))
    return fail(GNMR_E_INVALID, "out partly overlaps in (in place needs out == in)");
  const gnmr::ActSeg sg{static_cast<const char*>(in), static_cast<char*>(out), cols, unit};
  GNMR_HIP(gnmr::launch_actuate_matrix(sg, rows, d_mask, fmt_low, fmt_recovery,
                                       static_cast<hipStream_t>(stream)));
  return GNMR_OK;
}

gnmr_status gnmr_actuator_info(const gnmr_actuator* act, int64_t* rows, int64_t* bytes) {
  if (act == nullptr) return fail(GNMR_E_INVALID, "act is NULL");
  if (rows) *rows = act->rows;
  if (bytes) *bytes = act->bytes;
  return GNMR_OK;
}

gnmr_status gnmr_actuator_destroy(gnmr_actuator* act) {
  if (act == nullptr) return GNMR_OK;
  DeviceGuard g(act->device);
  if (act->arena) {
    (void)hipDeviceSynchronize();
    (void)hipFree(act->arena);
  }
  delete act;
  return GNMR_OK;
}

}  // extern "C"
