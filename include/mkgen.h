/*
 * mkgen.h -- seeded synthetic inputs for composed modules.
 *
 * A counter-based generator: element i of tensor t under seed s is a pure
 * function of (s, t, i), so the bytes do not depend on thread count or on
 * which slice of a tensor is generated.  It holds no arithmetic of the
 * modules themselves; the same bytes feed the HIP library and the oracle.
 *
 *   key  = mix64(s * 0x9E3779B97F4A7C15 + t)
 *   u_j  = mix64(key + j * 0x9E3779B97F4A7C15),  j = 2i + 1, 2i + 2
 *   U_j  = (u_j >> 11) * 2^-53                     in [0, 1)
 * where mix64 is the SplitMix64 output function (Steele, Lea and Flood,
 * "Fast splittable pseudorandom number generators", OOPSLA 2014).
 *   normal(mean, std):  mean + std * sqrt(-2 ln(1 - U_1)) * cos(2 pi U_2)   (Box-Muller)
 *   uniform(a, b):      a + (b - a) * U_1
 * The double is rounded to float32 (to nearest, ties to even) and, for a
 * bfloat16 tensor, the float32 is rounded to bfloat16 (ties to even).
 */
#ifndef MKGEN_H
#define MKGEN_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { MKGEN_NORMAL = 0, MKGEN_UNIFORM = 1 };
enum { MKGEN_F32 = 0, MKGEN_BF16 = 1 };

/* Fill elements [first, first + n) of tensor `tensor_id` into dst (host
   memory owned by the caller: n floats, or n uint16 bfloat16 bit patterns).
   dist: MKGEN_NORMAL (p0 = mean, p1 = std) or MKGEN_UNIFORM (p0 = a, p1 = b).
   Returns 0, or -1 on a bad argument (null dst, n < 0, unknown dist/dtype). */
int mkgen_fill(uint64_t seed, int32_t tensor_id, int32_t dist, double p0, double p1,
               int32_t dtype, int64_t first, int64_t n, void* dst);

#ifdef __cplusplus
}
#endif
#endif
