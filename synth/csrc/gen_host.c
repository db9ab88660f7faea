/* Host twin of the synthetic gradient generator (plain C, one thread per call).
 *
 * x(i) = rnd_dtype(scale * Z[j(i)]), j(i) = 16 bits of
 * SplitMix64(key + (i/4 + 1) * GAMMA) (Steele, Lea and Flood, OOPSLA 2014),
 * field i % 4.  Integer steps, one table lookup and one IEEE fp32 multiply:
 * bit-identical to synth/values.py and synth/csrc/gen.hip.  Build without
 * floating-point contraction or fast-math. */
#include <stdint.h>
#include <string.h>

static const uint64_t kGamma = 0x9E3779B97F4A7C15ull;

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

static inline uint16_t to_bf16(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static inline float value_at(uint64_t key, float scale, uint64_t i, const float* table) {
  const uint64_t h = mix64(key + ((i >> 2) + 1) * kGamma);
  return scale * table[(h >> (16 * (i & 3))) & 0xFFFFu];
}

/* Elements [start, start + count) of one unit; dtype 0 = fp32 (out: float[]),
 * 1 = bf16 (out: uint16_t[] bit patterns).  A ragged head and tail are done
 * one element at a time; full groups of four share one hash. */
void synth_host_values(uint64_t key, float scale, int dtype, int64_t start, int64_t count,
                       const float* table, void* out) {
  float* of = (float*)out;
  uint16_t* oh = (uint16_t*)out;
  int64_t k = 0;
  for (; k < count && ((start + k) & 3); ++k) {
    const float x = value_at(key, scale, (uint64_t)(start + k), table);
    if (dtype == 1) oh[k] = to_bf16(x);
    else of[k] = x;
  }
  const int64_t groups = (count - k) / 4;
  uint64_t g = (uint64_t)(start + k) >> 2;
  if (dtype == 1) {
    for (int64_t q = 0; q < groups; ++q, ++g, k += 4) {
      const uint64_t h = mix64(key + (g + 1) * kGamma);
      oh[k] = to_bf16(scale * table[h & 0xFFFFu]);
      oh[k + 1] = to_bf16(scale * table[(h >> 16) & 0xFFFFu]);
      oh[k + 2] = to_bf16(scale * table[(h >> 32) & 0xFFFFu]);
      oh[k + 3] = to_bf16(scale * table[(h >> 48) & 0xFFFFu]);
    }
  } else {
    for (int64_t q = 0; q < groups; ++q, ++g, k += 4) {
      const uint64_t h = mix64(key + (g + 1) * kGamma);
      of[k] = scale * table[h & 0xFFFFu];
      of[k + 1] = scale * table[(h >> 16) & 0xFFFFu];
      of[k + 2] = scale * table[(h >> 32) & 0xFFFFu];
      of[k + 3] = scale * table[(h >> 48) & 0xFFFFu];
    }
  }
  for (; k < count; ++k) {
    const float x = value_at(key, scale, (uint64_t)(start + k), table);
    if (dtype == 1) oh[k] = to_bf16(x);
    else of[k] = x;
  }
}
