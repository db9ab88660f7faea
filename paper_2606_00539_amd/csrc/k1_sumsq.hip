// K1 of the GNMR controller pass for CDNA4 (gfx950): the sum of squares of
// every gradient element, one fp32 partial per 64 KiB work item (Sec. 2,
// local-gradient equation: n = ||g||_2 over all of a unit's parameters).
//
// Deterministic: fixed work items, a fixed reduction tree, no floating-point
// atomics; the result does not depend on the grid or on scheduling.
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

// Streaming loads: every gradient byte is read exactly once, so the loads
// carry the non-temporal hint and do not displace cache lines worth keeping.
__device__ __forceinline__ u32x4 stream_load(const g_vec* p) {
  return __builtin_nontemporal_load(p);
}

// The 16-byte-aligned body of one item: lane i reads vectors i, i + 256, ...
// All 16 loads are issued before the first is consumed.  In a ragged item
// lanes past the end re-read the last vector (always in bounds) and add zero.
template <int DT>
__device__ __forceinline__ void body_sumsq(const g_vec* body, int nvec, int tid, float& a0,
                                           float& a1, float& a2, float& a3) {
  u32x4 v[kK1Unroll];
  if (nvec == kK1Block * kK1Unroll) {
#pragma unroll
    for (int k = 0; k < kK1Unroll; ++k) v[k] = stream_load(body + tid + k * kK1Block);
  } else if (nvec > 0) {
#pragma unroll
    for (int k = 0; k < kK1Unroll; ++k) {
      const int i = tid + k * kK1Block;
      v[k] = stream_load(body + (i < nvec ? i : nvec - 1));
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

// Workgroups are dispatched to the eight XCDs round-robin (workgroup w runs
// on XCD w % 8).  Give each XCD one contiguous eighth of the item list, so
// that each XCD's L2 and address translation see a single sequential stream.
// A bijection of [0, num_items) for any num_items.
__device__ __forceinline__ uint32_t xcd_item(uint32_t w, uint32_t num_items) {
  const uint32_t x = w % kNumXcd, j = w / kNumXcd;
  const uint32_t q = num_items / kNumXcd, r = num_items % kNumXcd;
  return x * q + (x < r ? x : r) + j;
}

__global__ __launch_bounds__(kK1Block) void k1_sumsq(const Item* __restrict__ items,
                                                     uint32_t num_items,
                                                     const char* const* __restrict__ seg_base,
                                                     const int32_t* __restrict__ seg_dtype,
                                                     float* __restrict__ partial) {
  const uint32_t item = xcd_item(blockIdx.x, num_items);
  const Item it = items[item];
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
  if (tid == 0) partial[item] = ((red[0] + red[1]) + red[2]) + red[3];
}

}  // namespace

hipError_t launch_sumsq(const Item* items, int64_t num_items, const char* const* seg_base,
                        const int32_t* seg_dtype, float* partial, hipStream_t s) {
  if (num_items <= 0) return hipSuccess;
  hipLaunchKernelGGL(k1_sumsq, dim3(unsigned(num_items)), dim3(kK1Block), 0, s, items,
                     uint32_t(num_items), seg_base, seg_dtype, partial);
  return hipGetLastError();
}

}  // namespace gnmr
