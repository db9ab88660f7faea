/* Oracle sum of squares in plain C -- TEST INFRASTRUCTURE ONLY (same rules
 * as the rest of oracle/: only tests, smoke and the CPU baseline use it).
 *
 * n_b^2 = sum_i g_i^2 (Sec. 2, local-gradient equation): each element is
 * widened exactly to double, squared exactly (bf16 and fp32 significands fit
 * in 53 bits twice over), and added in index order. */
#include <stdint.h>
#include <string.h>

double oracle_sumsq_f32(const float* x, int64_t n) {
  double s = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    const double v = (double)x[i];
    s += v * v;
  }
  return s;
}

double oracle_sumsq_bf16(const uint16_t* x, int64_t n) {
  double s = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    const uint32_t u = (uint32_t)x[i] << 16;
    float f;
    memcpy(&f, &u, 4);
    const double v = (double)f;
    s += v * v;
  }
  return s;
}
