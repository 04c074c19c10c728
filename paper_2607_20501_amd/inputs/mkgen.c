/* Seeded synthetic input generator; the definition is stated in mkgen.h. */
#include "../../include/mkgen.h"

#include <math.h>
#include <string.h>

static uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

static const uint64_t kGolden = 0x9E3779B97F4A7C15ull;

static uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

int mkgen_fill(uint64_t seed, int32_t tensor_id, int32_t dist, double p0, double p1,
               int32_t dtype, int64_t first, int64_t n, void* dst) {
  if (!dst || n < 0 || first < 0) return -1;
  if (dist != MKGEN_NORMAL && dist != MKGEN_UNIFORM) return -1;
  if (dtype != MKGEN_F32 && dtype != MKGEN_BF16) return -1;
  const uint64_t key = mix64(seed * kGolden + (uint64_t)(uint32_t)tensor_id);
  const double two_pi = 6.283185307179586476925286766559;
#pragma omp parallel for schedule(static)
  for (int64_t k = 0; k < n; ++k) {
    uint64_t i = (uint64_t)(first + k);
    double u1 = (double)(mix64(key + (2 * i + 1) * kGolden) >> 11) * 0x1.0p-53;
    double v;
    if (dist == MKGEN_NORMAL) {
      double u2 = (double)(mix64(key + (2 * i + 2) * kGolden) >> 11) * 0x1.0p-53;
      v = p0 + p1 * sqrt(-2.0 * log(1.0 - u1)) * cos(two_pi * u2);
    } else {
      v = p0 + (p1 - p0) * u1;
    }
    float f = (float)v;
    if (dtype == MKGEN_F32)
      ((float*)dst)[k] = f;
    else
      ((uint16_t*)dst)[k] = f32_to_bf16_rne(f);
  }
  return 0;
}
