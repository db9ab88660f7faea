// Synthetic gradient generator for gfx950 (test and benchmark harness only).
//
// Writes x(i) = rnd_dtype(s * Z[j(i)]) for every element i of a list of
// segments, with j(i) = 16 bits of SplitMix64(key + (i/4 + 1) * GAMMA)
// (Steele, Lea and Flood, OOPSLA 2014); key, s and the fp32 table Z come from
// the host.  Bit-identical to the NumPy host twin in synth/values.py.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

extern "C" {
typedef struct {
  void* ptr;           // device address of the segment's first element
  int64_t numel;       // elements in the segment
  int64_t unit_base;   // index of the segment's first element inside its unit
  uint64_t key;        // per-(seed, step, unit) key
  float scale;         // fp32 scale
  int32_t dtype;       // 0 = fp32, 1 = bf16
} synth_job;
}

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
constexpr int64_t kTile = int64_t(1) << 20;
constexpr int kBlock = 256;

struct Tile {
  int64_t job;
  int64_t start;
  int64_t count;
};

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__global__ __launch_bounds__(kBlock) void gen_kernel(const synth_job* __restrict__ jobs,
                                                     const Tile* __restrict__ tiles,
                                                     const float* __restrict__ table) {
  const Tile tl = tiles[blockIdx.x];
  const synth_job j = jobs[tl.job];
  const int64_t end = tl.start + tl.count;
  for (int64_t e = tl.start + threadIdx.x; e < end; e += kBlock) {
    const uint64_t i = uint64_t(j.unit_base + e);
    const uint64_t h = mix64(j.key + ((i >> 2) + 1) * kGamma);
    const uint32_t idx = uint32_t(h >> (16 * (i & 3))) & 0xFFFFu;
    const float x = __fmul_rn(j.scale, table[idx]);
    if (j.dtype == 1) {
      uint32_t u = __float_as_uint(x);
      u += 0x7FFFu + ((u >> 16) & 1u);
      static_cast<uint16_t*>(j.ptr)[e] = uint16_t(u >> 16);
    } else {
      static_cast<float*>(j.ptr)[e] = x;
    }
  }
}

}  // namespace

extern "C" {

// Fills every job's segment on `stream` and waits for it.  Returns 0, or the
// hipError_t of the first failing call.
int synth_fill(const synth_job* jobs, int64_t njobs, const float* d_table, void* stream) {
  if (njobs <= 0) return 0;
  hipStream_t st = static_cast<hipStream_t>(stream);
  std::vector<Tile> tiles;
  for (int64_t k = 0; k < njobs; ++k)
    for (int64_t s = 0; s < jobs[k].numel; s += kTile)
      tiles.push_back(Tile{k, s, jobs[k].numel - s < kTile ? jobs[k].numel - s : kTile});
  if (tiles.empty()) return 0;
  synth_job* d_jobs = nullptr;
  Tile* d_tiles = nullptr;
  hipError_t e = hipMalloc(&d_jobs, size_t(njobs) * sizeof(synth_job));
  if (e == hipSuccess) e = hipMalloc(&d_tiles, tiles.size() * sizeof(Tile));
  if (e == hipSuccess)
    e = hipMemcpyAsync(d_jobs, jobs, size_t(njobs) * sizeof(synth_job), hipMemcpyHostToDevice, st);
  if (e == hipSuccess)
    e = hipMemcpyAsync(d_tiles, tiles.data(), tiles.size() * sizeof(Tile), hipMemcpyHostToDevice,
                       st);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(gen_kernel, dim3(unsigned(tiles.size())), dim3(kBlock), 0, st, d_jobs,
                       d_tiles, d_table);
    e = hipGetLastError();
  }
  hipError_t e2 = hipStreamSynchronize(st);
  if (e == hipSuccess) e = e2;
  if (d_jobs) (void)hipFree(d_jobs);
  if (d_tiles) (void)hipFree(d_tiles);
  return int(e);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Read-ceiling probes (benchmark reference points, not part of the method):
// plain read-reduce kernels over a contiguous 16-byte-aligned buffer, each
// lane summing the fp32 squares of the words it reads, one fp32 partial per
// workgroup.  They show the read rate a minimal kernel reaches on the same
// bytes as the gradient pass.
// ---------------------------------------------------------------------------
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const u32x4 g_vec;
constexpr int kProbeUnroll = 16;
constexpr int64_t kProbeBlockVecs = int64_t(kBlock) * kProbeUnroll;   // 64 KiB per workgroup

__device__ __forceinline__ float sq4(const u32x4& v) {
  float a = __uint_as_float(v.x), b = __uint_as_float(v.y), c = __uint_as_float(v.z),
        d = __uint_as_float(v.w);
  return (a * a + b * b) + (c * c + d * d);
}

__device__ __forceinline__ void block_partial(float s, float* out) {
  __shared__ float red[kBlock / 64];
  for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) out[blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
}

// Variant 0: grid-stride loop, 16-byte non-temporal loads, 8 in flight per lane.
__global__ __launch_bounds__(kBlock) void probe_grid_stride(const g_vec* __restrict__ p,
                                                            int64_t nvec, float* out) {
  const int64_t stride = int64_t(gridDim.x) * kBlock;
  float s = 0.f;
  int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  for (; i + 7 * stride < nvec; i += 8 * stride) {
    u32x4 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = __builtin_nontemporal_load(p + i + k * stride);
#pragma unroll
    for (int k = 0; k < 8; ++k) s += sq4(v[k]);
  }
  for (; i < nvec; i += stride) s += sq4(__builtin_nontemporal_load(p + i));
  block_partial(s, out);
}

// Variant 1: one 64 KiB block per workgroup, all 16 loads of a lane issued
// before the first is used, blocks dealt to the eight XCDs in contiguous
// runs (workgroup w runs on XCD w % 8) -- the gradient pass's read pattern
// without its work-item table.
__global__ __launch_bounds__(kBlock) void probe_blocked(const g_vec* __restrict__ p, int64_t nvec,
                                                        float* out) {
  const uint32_t nblk = gridDim.x, w = blockIdx.x;
  const uint32_t x = w % 8, j = w / 8, q = nblk / 8, r = nblk % 8;
  const int64_t blk = int64_t(x) * q + (x < r ? x : r) + j;
  const int64_t v0 = blk * kProbeBlockVecs;
  const int64_t n = nvec - v0 < kProbeBlockVecs ? nvec - v0 : kProbeBlockVecs;
  u32x4 v[kProbeUnroll];
#pragma unroll
  for (int k = 0; k < kProbeUnroll; ++k) {
    const int64_t i = threadIdx.x + int64_t(k) * kBlock;
    v[k] = __builtin_nontemporal_load(p + v0 + (i < n ? i : n - 1));
  }
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < kProbeUnroll; ++k)
    if (threadIdx.x + int64_t(k) * kBlock < n) s += sq4(v[k]);
  block_partial(s, out);
}

}  // namespace

extern "C" {

// Number of fp32 partials synth_read_probe writes for `bytes` and `variant`.
int64_t synth_read_probe_partials(int64_t bytes, int32_t variant) {
  const int64_t nvec = bytes / 16;
  if (nvec <= 0) return 0;
  return variant == 0 ? int64_t(256) * 8 : (nvec + kProbeBlockVecs - 1) / kProbeBlockVecs;
}

// Launches one read-reduce pass over `bytes` (a multiple of 16) at the
// 16-byte-aligned device address `p` on `stream`; `partials` holds
// synth_read_probe_partials(bytes, variant) floats.  Returns 0 or a hipError_t
// (1 = hipErrorInvalidValue for bad arguments).
int synth_read_probe(const void* p, int64_t bytes, float* partials, int32_t variant,
                     void* stream) {
  if (p == nullptr || partials == nullptr || bytes <= 0 || bytes % 16 != 0 ||
      reinterpret_cast<uintptr_t>(p) % 16 != 0 || (variant != 0 && variant != 1))
    return int(hipErrorInvalidValue);
  const int64_t nvec = bytes / 16;
  const int64_t grid = synth_read_probe_partials(bytes, variant);
  if (grid > int64_t(UINT32_MAX)) return int(hipErrorInvalidValue);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (variant == 0)
    hipLaunchKernelGGL(probe_grid_stride, dim3(unsigned(grid)), dim3(kBlock), 0, st,
                       (const g_vec*)reinterpret_cast<uintptr_t>(p), nvec, partials);
  else
    hipLaunchKernelGGL(probe_blocked, dim3(unsigned(grid)), dim3(kBlock), 0, st,
                       (const g_vec*)reinterpret_cast<uintptr_t>(p), nvec, partials);
  return int(hipGetLastError());
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Read-and-write reference: a plain copy of `bytes` (a multiple of 16) from
// src to dst, 4 non-temporal 16-byte loads then 4 non-temporal stores per
// lane, one 16 KiB block per workgroup in XCD-contiguous order (the best of
// a sweep of block sizes on this part).  A reference point for kernels that
// read and write every byte once.
// ---------------------------------------------------------------------------
namespace {

typedef __attribute__((address_space(1))) u32x4 g_vec_w;
constexpr int kCopyUnroll = 4;
constexpr int64_t kCopyBlockVecs = int64_t(kBlock) * kCopyUnroll;

__global__ __launch_bounds__(kBlock) void probe_copy(const g_vec* __restrict__ src,
                                                     g_vec_w* __restrict__ dst, int64_t nvec) {
  const uint32_t nblk = gridDim.x, w = blockIdx.x;
  const uint32_t x = w % 8, j = w / 8, q = nblk / 8, r = nblk % 8;
  const int64_t v0 = (int64_t(x) * q + (x < r ? x : r) + j) * kCopyBlockVecs;
  u32x4 v[kCopyUnroll];
#pragma unroll
  for (int k = 0; k < kCopyUnroll; ++k) {
    const int64_t i = v0 + threadIdx.x + int64_t(k) * kBlock;
    if (i < nvec) v[k] = __builtin_nontemporal_load(src + i);
  }
#pragma unroll
  for (int k = 0; k < kCopyUnroll; ++k) {
    const int64_t i = v0 + threadIdx.x + int64_t(k) * kBlock;
    if (i < nvec) __builtin_nontemporal_store(v[k], dst + i);
  }
}

}  // namespace

extern "C" {

// Launches one copy on `stream`; both addresses 16-byte aligned, the ranges
// disjoint.  Returns 0 or a hipError_t (1 = hipErrorInvalidValue).
int synth_copy_probe(const void* src, void* dst, int64_t bytes, void* stream) {
  if (src == nullptr || dst == nullptr || bytes <= 0 || bytes % 16 != 0 ||
      (reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) % 16 != 0)
    return int(hipErrorInvalidValue);
  const int64_t nvec = bytes / 16;
  const int64_t grid = (nvec + kCopyBlockVecs - 1) / kCopyBlockVecs;
  if (grid > int64_t(UINT32_MAX)) return int(hipErrorInvalidValue);
  hipLaunchKernelGGL(probe_copy, dim3(unsigned(grid)), dim3(kBlock), 0,
                     static_cast<hipStream_t>(stream),
                     (const g_vec*)reinterpret_cast<uintptr_t>(src),
                     (g_vec_w*)reinterpret_cast<uintptr_t>(dst), nvec);
  return int(hipGetLastError());
}

}  // extern "C"
