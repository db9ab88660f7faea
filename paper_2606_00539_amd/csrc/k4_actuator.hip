// K4, the recovery actuator for CDNA4 (gfx950): per-token fake quantisation
// of saved activations, the format chosen per unit by the controller's mask
// (App. E.2 quantisation-simulated operators: each token is scaled into the
// format's representable range, rounded to the nearest representable value
// and rescaled; Sec. 5.1 / App. E.4: token-wise low-bit saved activations;
// Sec. 5.3 / App. E.3: the INT8 low-cost path).
//
// One wavefront per token row of up to 4096 features, one workgroup per
// longer row (up to 16384), the row held in registers: amax by a
// max-reduction, one fp32 division each for the scale and its reciprocal,
// then per element y = x * inv, round to the format (ties to the even
// significand, saturating), out = bf16_rne(q * s).  A row whose unit takes
// the BF16 path in place is left untouched without reading it.  The rows come
// from a table built once over many segments (k4_actuate*), or from one
// matrix passed by value (k4_matrix*, no table).  Rows are
// dealt to the eight XCDs in contiguous runs, and both loads and stores are
// non-temporal: every byte is read and written once.
#include "gnmr_internal.h"

namespace gnmr {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const u32x4 g_cvec;
typedef __attribute__((address_space(1))) u32x4 g_vec;

struct Format {
  int mbits;    // significand bits
  int emin;     // exponent of the smallest normal binade
  float fmax;   // largest finite value
};

// E2M1, E3M2, E4M3 (OCP, 448 max), E5M2 (57344 max); no inf/NaN produced.
// The symmetric INT8 grid {0, 1, ..., 127} is the same rounding with the
// lowest binade at 2^6 and 6 fraction bits: a step of 1 below 128 and
// saturation at 127.
__device__ __forceinline__ Format format_of(int fmt) {
  switch (fmt) {
    case GNMR_FMT_INT8: return Format{6, 6, 127.0f};
    case GNMR_FMT_E2M1: return Format{1, 0, 6.0f};
    case GNMR_FMT_E3M2: return Format{2, -2, 28.0f};
    case GNMR_FMT_E4M3: return Format{3, -6, 448.0f};
    default: return Format{2, -14, 57344.0f};  // GNMR_FMT_E5M2
  }
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two fp32 values to packed bf16, round to nearest even (one
// v_cvt_pk_bf16_f32; the values here are finite).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// Nearest representable value of the format to y, ties to the even
// significand, saturating at fmax.  All steps but rintf are exact.
__device__ __forceinline__ float round_to_format(float y, const Format& f) {
  const float a = fabsf(y);
  int e = int((__float_as_uint(a) >> 23) & 0xFFu) - 127;  // binade of a (any e < emin clamps)
  e = e < f.emin ? f.emin : e;
  const float step = __uint_as_float(uint32_t(e - f.mbits + 127) << 23);
  const float inv_step = __uint_as_float(uint32_t(f.mbits - e + 127) << 23);
  float q = __fmul_rn(rintf(__fmul_rn(a, inv_step)), step);
  q = q < f.fmax ? q : f.fmax;
  return copysignf(q, y);
}

__device__ __forceinline__ uint32_t quant_pair(uint32_t w, float inv, float s, const Format& f) {
  const float lo = __fmul_rn(round_to_format(__fmul_rn(bf16_lo(w), inv), f), s);
  const float hi = __fmul_rn(round_to_format(__fmul_rn(bf16_hi(w), inv), f), s);
  return pack_bf16(lo, hi);
}

__device__ __forceinline__ float max_abs_pair(uint32_t w, float m) {
  return fmaxf(m, fmaxf(fabsf(bf16_lo(w)), fabsf(bf16_hi(w))));
}

__device__ __forceinline__ void store(g_vec* p, const u32x4& v) {
  __builtin_nontemporal_store(v, p);
}

// Row `row` of segment sg by LANES lanes (64: a wavefront; kK4Block: the
// workgroup).  Every lane of the group calls it; `red` is workgroup LDS when
// LANES > 64.
template <int LANES>
__device__ __forceinline__ void actuate_row(const ActSeg sg, int64_t row,
                                            const uint8_t* __restrict__ mask, int fmt_low,
                                            int fmt_rec, int lane, float* red) {
  const int fmt = mask[sg.unit] ? fmt_rec : fmt_low;
  const int64_t row_off = row * sg.cols * 2;
  if (fmt == GNMR_FMT_BF16 && sg.in == sg.out) return;  // BF16 path in place: nothing to do
  const g_cvec* in = (const g_cvec*)(sg.in + row_off);
  g_vec* out = (g_vec*)(sg.out + row_off);
  const int nvec = sg.cols >> 3;

  u32x4 v[kK4Vpt];
#pragma unroll
  for (int k = 0; k < kK4Vpt; ++k) {
    const int i = lane + k * LANES;
    v[k] = i < nvec ? __builtin_nontemporal_load(in + i) : u32x4{0u, 0u, 0u, 0u};
  }
  if (fmt == GNMR_FMT_BF16) {  // BF16 path out of place: a copy
#pragma unroll
    for (int k = 0; k < kK4Vpt; ++k) {
      const int i = lane + k * LANES;
      if (i < nvec) store(out + i, v[k]);
    }
    return;
  }

  // amax over the row (max is exact, so the reduction order is immaterial)
  float m = 0.0f;
#pragma unroll
  for (int k = 0; k < kK4Vpt; ++k) {
    m = max_abs_pair(v[k].x, m);
    m = max_abs_pair(v[k].y, m);
    m = max_abs_pair(v[k].z, m);
    m = max_abs_pair(v[k].w, m);
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) m = fmaxf(m, __shfl_xor(m, d, 64));
  float amax = m;
  if constexpr (LANES > 64) {
    static_assert(LANES == 4 * 64, "four waves per row");
    if ((lane & 63) == 0) red[lane >> 6] = m;
    __syncthreads();
    amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  }

  const Format f = format_of(fmt);
  if (amax == 0.0f) {  // an all-zero token stays zero
#pragma unroll
    for (int k = 0; k < kK4Vpt; ++k) {
      const int i = lane + k * LANES;
      if (i < nvec) store(out + i, u32x4{0u, 0u, 0u, 0u});
    }
    return;
  }
  const float inv = __fdiv_rn(f.fmax, amax);  // scale into the format's range
  const float s = __fdiv_rn(amax, f.fmax);    // and back
#pragma unroll
  for (int k = 0; k < kK4Vpt; ++k) {
    const int i = lane + k * LANES;
    if (i < nvec) {
      u32x4 o;
      o.x = quant_pair(v[k].x, inv, s, f);
      o.y = quant_pair(v[k].y, inv, s, f);
      o.z = quant_pair(v[k].z, inv, s, f);
      o.w = quant_pair(v[k].w, inv, s, f);
      store(out + i, o);
    }
  }
}

// Workgroup w runs on XCD w % 8: give each XCD a contiguous run of [0, n).
__device__ __forceinline__ uint32_t xcd_order(uint32_t w, uint32_t n) {
  const uint32_t x = w % kNumXcd, j = w / kNumXcd, q = n / kNumXcd, r = n % kNumXcd;
  return x * q + (x < r ? x : r) + j;
}

// At most 80 VGPRs (six waves per SIMD): more rows in flight per CU.
__global__ __launch_bounds__(kK4Block) __attribute__((amdgpu_waves_per_eu(6, 8))) void
k4_actuate_wave(const RowItem* __restrict__ items, uint32_t num_rows,
                const ActSeg* __restrict__ segs, const uint8_t* __restrict__ mask, int fmt_low,
                int fmt_rec) {
  const uint32_t rows_per_wg = kK4Block / 64;
  const uint32_t r = xcd_order(blockIdx.x, gridDim.x) * rows_per_wg + (threadIdx.x >> 6);
  if (r >= num_rows) return;
  const RowItem it = items[r];
  actuate_row<64>(segs[it.seg], it.row, mask, fmt_low, fmt_rec, int(threadIdx.x & 63), nullptr);
}

__global__ __launch_bounds__(kK4Block) __attribute__((amdgpu_waves_per_eu(6, 8))) void
k4_actuate(const RowItem* __restrict__ items, const ActSeg* __restrict__ segs,
           const uint8_t* __restrict__ mask, int fmt_low, int fmt_rec) {
  __shared__ float red[kK4Block / 64];
  const RowItem it = items[xcd_order(blockIdx.x, gridDim.x)];
  actuate_row<kK4Block>(segs[it.seg], it.row, mask, fmt_low, fmt_rec, int(threadIdx.x), red);
}

// One matrix without a row table (the segment passed by value): rows of at
// most kK4WaveCols features, four per workgroup, one wavefront each.
__global__ __launch_bounds__(kK4Block) __attribute__((amdgpu_waves_per_eu(6, 8))) void
k4_matrix_wave(const ActSeg sg, int64_t num_rows, const uint8_t* __restrict__ mask, int fmt_low,
               int fmt_rec) {
  const int64_t r =
      int64_t(xcd_order(blockIdx.x, gridDim.x)) * (kK4Block / 64) + (threadIdx.x >> 6);
  if (r >= num_rows) return;
  actuate_row<64>(sg, r, mask, fmt_low, fmt_rec, int(threadIdx.x & 63), nullptr);
}

// One matrix without a row table, rows longer than kK4WaveCols: one
// workgroup per row.
__global__ __launch_bounds__(kK4Block) __attribute__((amdgpu_waves_per_eu(6, 8))) void
k4_matrix(const ActSeg sg, const uint8_t* __restrict__ mask, int fmt_low, int fmt_rec) {
  __shared__ float red[kK4Block / 64];
  actuate_row<kK4Block>(sg, xcd_order(blockIdx.x, gridDim.x), mask, fmt_low, fmt_rec,
                        int(threadIdx.x), red);
}

}  // namespace

hipError_t launch_actuate(const RowItem* items, int64_t num_narrow, int64_t num_rows,
                          const ActSeg* segs, const uint8_t* mask, int fmt_low, int fmt_rec,
                          hipStream_t s) {
  const int64_t rows_per_wg = kK4Block / 64;
  if (num_narrow > 0)
    hipLaunchKernelGGL(k4_actuate_wave, dim3(unsigned((num_narrow + rows_per_wg - 1) / rows_per_wg)),
                       dim3(kK4Block), 0, s, items, uint32_t(num_narrow), segs, mask, fmt_low,
                       fmt_rec);
  if (num_rows > num_narrow)
    hipLaunchKernelGGL(k4_actuate, dim3(unsigned(num_rows - num_narrow)), dim3(kK4Block), 0, s,
                       items + num_narrow, segs, mask, fmt_low, fmt_rec);
  return hipGetLastError();
}

hipError_t launch_actuate_matrix(const ActSeg& sg, int64_t rows, const uint8_t* mask,
                                 int fmt_low, int fmt_rec, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (sg.cols <= kK4WaveCols) {
    const int64_t rows_per_wg = kK4Block / 64;
    hipLaunchKernelGGL(k4_matrix_wave, dim3(unsigned((rows + rows_per_wg - 1) / rows_per_wg)),
                       dim3(kK4Block), 0, s, sg, rows, mask, fmt_low, fmt_rec);
  } else {
    hipLaunchKernelGGL(k4_matrix, dim3(unsigned(rows)), dim3(kK4Block), 0, s, sg, mask, fmt_low,
                       fmt_rec);
  }
  return hipGetLastError();
}

}  // namespace gnmr
