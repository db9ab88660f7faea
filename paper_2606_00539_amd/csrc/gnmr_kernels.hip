// Kernels of the GNMR controller pass for CDNA4 (gfx950).
//
//   K1 k1_sumsq        sum of squares of every gradient element, one fp32
//                      partial per 64 KiB work item (Sec. 2, local-gradient
//                      equation: n = ||g||_2 over all of a unit's parameters)
//   K2 k2_update       per unit: fixed-order float64 sum of its partials,
//                      n = sqrt, then Alg. 1 (GNMR, Delta-GNMR, running mean,
//                      queue) and the risk R of Alg. 2
//   K3 k3_select       one workgroup: candidate pool, Top_maxO by R (ties to
//                      the smaller index), lock update and step counters
//                      (Alg. 2; Sec. 3.3, 3.4)
//
// Everything is deterministic: fixed work items, fixed reduction trees, no
// floating-point atomics.
#include <math.h>

#include "gnmr_internal.h"

namespace gnmr {
namespace {

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Butterfly over the 64 lanes of a wavefront; every lane ends with the same sum.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// One 16-byte load as a native vector (loads through address-space-1
// pointers need a plain vector type, not HIP's uint4 class).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Eight bf16 values of one 16-byte load; two squares into each accumulator.
__device__ __forceinline__ void acc_bf16(const u32x4& x, float& a0, float& a1, float& a2,
                                         float& a3) {
  float v;
  v = bf16_lo(x.x); a0 = fmaf(v, v, a0);
  v = bf16_hi(x.x); a1 = fmaf(v, v, a1);
  v = bf16_lo(x.y); a2 = fmaf(v, v, a2);
  v = bf16_hi(x.y); a3 = fmaf(v, v, a3);
  v = bf16_lo(x.z); a0 = fmaf(v, v, a0);
  v = bf16_hi(x.z); a1 = fmaf(v, v, a1);
  v = bf16_lo(x.w); a2 = fmaf(v, v, a2);
  v = bf16_hi(x.w); a3 = fmaf(v, v, a3);
}

// Four fp32 values of one 16-byte load.
__device__ __forceinline__ void acc_f32(const u32x4& x, float& a0, float& a1, float& a2,
                                        float& a3) {
  float v;
  v = __uint_as_float(x.x); a0 = fmaf(v, v, a0);
  v = __uint_as_float(x.y); a1 = fmaf(v, v, a1);
  v = __uint_as_float(x.z); a2 = fmaf(v, v, a2);
  v = __uint_as_float(x.w); a3 = fmaf(v, v, a3);
}

template <int DT>
__device__ __forceinline__ void acc_vec(const u32x4& x, float& a0, float& a1, float& a2,
                                        float& a3) {
  if constexpr (DT == GNMR_BF16) acc_bf16(x, a0, a1, a2, a3);
  else acc_f32(x, a0, a1, a2, a3);
}

// Global-address-space views, so that the loads are global_load (not flat).
typedef __attribute__((address_space(1))) const u32x4 g_vec;
typedef __attribute__((address_space(1))) const uint16_t g_u16;
typedef __attribute__((address_space(1))) const float g_f32;

// The 16-byte-aligned body of one item: lane i reads vectors i, i + 256, ...
// All 16 loads are issued before the first is consumed.  In a ragged item
// lanes past the end re-read the last vector (always in bounds) and add zero.
template <int DT>
__device__ __forceinline__ void body_sumsq(const g_vec* body, int nvec, int tid, float& a0,
                                           float& a1, float& a2, float& a3) {
  u32x4 v[kK1Unroll];
  if (nvec == kK1Block * kK1Unroll) {
#pragma unroll
    for (int k = 0; k < kK1Unroll; ++k) v[k] = body[tid + k * kK1Block];
  } else if (nvec > 0) {
#pragma unroll
    for (int k = 0; k < kK1Unroll; ++k) {
      const int i = tid + k * kK1Block;
      v[k] = body[i < nvec ? i : nvec - 1];
    }
#pragma unroll
    for (int k = 0; k < kK1Unroll; ++k)
      if (tid + k * kK1Block >= nvec) v[k] = u32x4{0u, 0u, 0u, 0u};
  } else {
    return;
  }
#pragma unroll
  for (int k = 0; k < kK1Unroll; ++k) acc_vec<DT>(v[k], a0, a1, a2, a3);
}

__global__ __launch_bounds__(kK1Block) void k1_sumsq(const Item* __restrict__ items,
                                                     const char* const* __restrict__ seg_base,
                                                     const int32_t* __restrict__ seg_dtype,
                                                     float* __restrict__ partial) {
  const Item it = items[blockIdx.x];
  const int dt = seg_dtype[it.seg];
  const uintptr_t esz = dt == GNMR_BF16 ? 2 : 4;
  const uintptr_t b0 = reinterpret_cast<uintptr_t>(seg_base[it.seg]) + uintptr_t(it.e0) * esz;
  const uintptr_t b1 = b0 + uintptr_t(it.count) * esz;
  // [b0, a0) head and [a1, b1) tail are under 16 bytes each; [a0, a1) is the
  // 16-byte-aligned body.  An item inside one 16-byte window is all head.
  uintptr_t a0 = (b0 + 15) & ~uintptr_t(15);
  uintptr_t a1 = b1 & ~uintptr_t(15);
  if (a0 > a1) a0 = a1 = b1;
  const int nvec = int((a1 - a0) >> 4);
  const int tid = threadIdx.x;
  const g_vec* body = (const g_vec*)a0;

  float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
  if (dt == GNMR_BF16) body_sumsq<GNMR_BF16>(body, nvec, tid, s0, s1, s2, s3);
  else body_sumsq<GNMR_F32>(body, nvec, tid, s0, s1, s2, s3);

  // head: lanes 0..7, tail: lanes 8..15, one element each at most
  uintptr_t e = 0;
  bool have = false;
  if (tid < 8) {
    e = b0 + uintptr_t(tid) * esz;
    have = e < a0;
  } else if (tid < 16) {
    e = a1 + uintptr_t(tid - 8) * esz;
    have = e < b1;
  }
  if (have) {
    const float v = dt == GNMR_BF16 ? __uint_as_float(uint32_t(*(const g_u16*)e) << 16)
                                    : *(const g_f32*)e;
    s0 = fmaf(v, v, s0);
  }

  float s = (s0 + s1) + (s2 + s3);
  s = wave_sum(s);
  __shared__ float red[kK1Block / 64];
  if ((tid & 63) == 0) red[tid >> 6] = s;
  __syncthreads();
  if (tid == 0) partial[blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
}

// Fixed-order float64 sum of unit b's item partials by one wavefront.
__device__ __forceinline__ double unit_ss(const int64_t* __restrict__ off,
                                          const float* __restrict__ partial, int b, int lane) {
  double s = 0.0;
  const int64_t hi = off[b + 1];
  for (int64_t i = off[b] + lane; i < hi; i += 64) s += double(partial[i]);
  return wave_sum(s);
}

__global__ __launch_bounds__(256) void k_unit_sumsq(const int64_t* __restrict__ off,
                                                    const float* __restrict__ partial,
                                                    int num_units, double* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= num_units) return;
  const double s = unit_ss(off, partial, b, lane);
  if (lane == 0) out[b] = s;
}

// K2: one wavefront per unit.
__global__ __launch_bounds__(256) void k2_update(UpdateArgs a) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= a.num_units) return;
  double n;
  if (a.ext_norm != nullptr) {
    n = a.ext_norm[b];
  } else {
    n = sqrt(unit_ss(a.unit_item_off, a.partial, b, lane));
  }
  if (lane != 0) return;

  const int U = a.num_units;
  const bool finite = isfinite(n);
  const double A_prev = a.A[b];
  // Alg. 1: GNMR = 1 at t = 1 or while the historical mean is 0.
  double G = 1.0;
  if (finite && a.t > 1 && A_prev != 0.0) G = n / (A_prev + a.eps);
  // Alg. 1: Delta-GNMR once the queue holds delta values, oldest first.
  double D = 1.0;
  if (a.qlen == a.window) {
    double total = 0.0;
    int slot = a.slot;
    for (int j = 0; j < a.window; ++j) {
      total += a.Q[int64_t(slot) * U + b];
      slot = slot + 1 == a.window ? 0 : slot + 1;
    }
    const double den = total / double(a.window) + a.eps;
    if (finite && den != 0.0) D = G / den;
  }
  // Alg. 1: running mean and queue push (the new value replaces the oldest).
  if (finite) a.A[b] = A_prev + (n - A_prev) / double(a.t);
  a.Q[int64_t(a.slot) * U + b] = finite ? G : 1.0;
  if (!finite) G = D = INFINITY;

  // Alg. 2: R = max(GNMR / alpha, Delta-GNMR / beta).
  const double gt = G / a.alpha;
  const double dt = D / a.beta;
  const double R = gt > dt ? gt : dt;
  a.norm[b] = n;
  a.gnmr[b] = G;
  a.dgnmr[b] = D;
  a.risk[b] = R;
  a.flags[b] = uint8_t((gt > 1.0 ? kFlagTrigG : 0) | (dt > 1.0 ? kFlagTrigD : 0) |
                       (finite ? 0 : kFlagNonFinite));
}

constexpr int kK3Block = 1024;

// Order-preserving key of a candidate: R >= 0 (or +inf), so its IEEE bits
// are monotone in R; +1 keeps 0 free for "not a candidate".
__device__ __forceinline__ uint64_t cand_key(double R) {
  return uint64_t(__double_as_longlong(R)) + 1;
}

// K3: a single workgroup.  Top_maxO is a radix select over the 64-bit keys
// (8 passes of 8 bits, most significant first) for the maxO-th largest key
// T; then every candidate with key > T is active, and the first `need`
// candidates with key == T in index order.
__global__ __launch_bounds__(kK3Block) void k3_select(SelectArgs a, uint64_t* __restrict__ keys) {
  __shared__ int cnt[6];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t scan[kK3Block];
  __shared__ int s_digit, s_k;
  const int tid = threadIdx.x;
  const int U = a.num_units;
  if (tid < 6) cnt[tid] = 0;
  __syncthreads();

  int c_cand = 0, c_tg = 0, c_td = 0, c_tr = 0, c_nf = 0;
  for (int b = tid; b < U; b += kK3Block) {
    const double R = a.risk[b];
    const uint8_t f = a.flags[b];
    const bool rec = a.rec[b] != 0;
    const bool trig = R > 1.0;
    const bool cand = rec && (trig || a.lock[b] > 0);
    keys[b] = cand ? cand_key(R) : 0;
    c_cand += cand;
    if (rec) {
      c_tg += (f & kFlagTrigG) != 0;
      c_td += (f & kFlagTrigD) != 0;
      c_tr += trig;
    }
    c_nf += (f & kFlagNonFinite) != 0;
  }
  atomicAdd(&cnt[0], c_cand);
  atomicAdd(&cnt[1], c_tg);
  atomicAdd(&cnt[2], c_td);
  atomicAdd(&cnt[3], c_tr);
  atomicAdd(&cnt[4], c_nf);
  __syncthreads();
  const int n_cand = cnt[0];

  uint64_t T;       // threshold key
  int need = 0;     // how many keys equal to T to take, in index order
  if (a.max_o == 0) {
    T = ~uint64_t(0);
  } else if (n_cand <= a.max_o) {
    T = 0;          // every candidate (key >= 1)
  } else {
    uint64_t prefix = 0, pmask = 0;
    int k = a.max_o;  // rank of T from the top, 1-based
    for (int shift = 56; shift >= 0; shift -= 8) {
      if (tid < 256) hist[tid] = 0;
      __syncthreads();
      for (int b = tid; b < U; b += kK3Block) {
        const uint64_t key = keys[b];
        if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (tid == 0) {
        uint32_t cum = 0;
        int d = 255;
        for (; d > 0; --d) {
          if (cum + hist[d] >= uint32_t(k)) break;
          cum += hist[d];
        }
        s_digit = d;
        s_k = k - int(cum);
      }
      __syncthreads();
      prefix |= uint64_t(s_digit) << shift;
      pmask |= uint64_t(255) << shift;
      k = s_k;
      __syncthreads();
    }
    T = prefix;
    need = k;
  }

  // Final pass over contiguous index ranges so that ties at T are ranked in
  // index order: exclusive scan of per-thread tie counts.
  const int per = (U + kK3Block - 1) / kK3Block;
  const int lo = tid * per < U ? tid * per : U;
  const int hi = lo + per < U ? lo + per : U;
  uint32_t ties = 0;
  if (need > 0)
    for (int b = lo; b < hi; ++b) ties += keys[b] == T;
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
    const uint64_t key = keys[b];
    bool sel = key > T;
    if (!sel && need > 0 && key == T) {
      sel = rank < uint32_t(need);
      ++rank;
    }
    int32_t L = 0;
    if (sel) {
      const int32_t prev = a.lock[b];
      L = a.risk[b] > 1.0 ? a.lock_len : (prev > 0 ? prev - 1 : 0);
    }
    a.lock[b] = L;
    a.mask[b] = sel ? 1 : 0;
    c_act += sel;
  }
  atomicAdd(&cnt[5], c_act);
  __syncthreads();
  if (tid == 0) {
    gnmr_stats st;
    st.t = a.t;
    st.n_trig_gnmr = cnt[1];
    st.n_trig_dgnmr = cnt[2];
    st.n_trig = cnt[3];
    st.n_cand = n_cand;
    st.n_active = cnt[5];
    st.hit_maxo = (n_cand > 0 && n_cand >= a.max_o) ? 1 : 0;
    st.n_nonfinite = cnt[4];
    st.reserved = 0;
    *a.stats = st;
  }
}

}  // namespace

hipError_t launch_sumsq(const Item* items, int64_t num_items, const char* const* seg_base,
                        const int32_t* seg_dtype, float* partial, hipStream_t s) {
  if (num_items <= 0) return hipSuccess;
  hipLaunchKernelGGL(k1_sumsq, dim3(unsigned(num_items)), dim3(kK1Block), 0, s, items, seg_base,
                     seg_dtype, partial);
  return hipGetLastError();
}

hipError_t launch_unit_sumsq(const int64_t* unit_item_off, const float* partial,
                             int32_t num_units, double* out, hipStream_t s) {
  hipLaunchKernelGGL(k_unit_sumsq, dim3(unsigned((num_units + 3) / 4)), dim3(256), 0, s,
                     unit_item_off, partial, num_units, out);
  return hipGetLastError();
}

hipError_t launch_update(const UpdateArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k2_update, dim3(unsigned((a.num_units + 3) / 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_select(const SelectArgs& a, uint64_t* keys, hipStream_t s) {
  hipLaunchKernelGGL(k3_select, dim3(1), dim3(kK3Block), 0, s, a, keys);
  return hipGetLastError();
}

}  // namespace gnmr
