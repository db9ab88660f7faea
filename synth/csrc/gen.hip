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
