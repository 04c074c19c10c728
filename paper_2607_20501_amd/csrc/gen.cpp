// mk_gen_fill: the seeded input generator (include/mkgen.h, compiled from
// inputs/mkgen.c into this library) behind the library's C ABI.  It holds none
// of the modules' arithmetic.
#include "../../include/mk.h"
#include "../../include/mkgen.h"
#include "plan.hpp"

extern "C" mk_status mk_gen_fill(uint64_t seed, int32_t tensor_id, int32_t dist, double p0,
                                 double p1, int32_t dtype, void* host_dst, int64_t n) {
  if (dtype != MK_F32 && dtype != MK_BF16) return mk::fail(MK_E_DTYPE, "mk_gen_fill: dtype");
  if (n < 0 || (n > 0 && !host_dst) || (dist != MKGEN_NORMAL && dist != MKGEN_UNIFORM))
    return mk::fail(MK_E_INVALID_ARG, "mk_gen_fill: null destination, n < 0 or unknown dist");
  if (n == 0) return MK_OK;
  const int32_t gdt = dtype == MK_BF16 ? MKGEN_BF16 : MKGEN_F32;
  if (mkgen_fill(seed, tensor_id, dist, p0, p1, gdt, 0, n, host_dst) != 0)
    return mk::fail(MK_E_INVALID_ARG, "mk_gen_fill: rejected arguments");
  return MK_OK;
}
