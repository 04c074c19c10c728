// Unsigned 32-bit division by a run-time divisor d >= 1 as one multiply-high,
// one add and one shift: the round-up method of Granlund & Montgomery
// ("Division by invariant integers using multiplication", PLDI 1994, Thm. 4.2).
// With s = ceil(log2 d) and m = floor(2^32 (2^s - d) / d) + 1,
//   n / d = (mulhi32(n, m) + n) >> s    for every n < 2^32,
// the sum taken in 64 bits so it cannot wrap.  Plain C++ (the members are
// constexpr, which HIP also compiles for the device), so the host test suite
// checks it against the '/' operator.
#pragma once
#include <cstdint>

namespace mk {

struct FastDiv {
  uint32_t d = 1, m = 1, s = 0;

  FastDiv() = default;
  constexpr explicit FastDiv(uint32_t divisor) : d(divisor), m(1), s(0) {
    while (s < 32 && (uint64_t(1) << s) < divisor) ++s;
    m = (uint32_t)(((uint64_t(1) << 32) * ((uint64_t(1) << s) - divisor)) / divisor + 1);
  }
  constexpr uint32_t div(uint32_t n) const {
    return (uint32_t)((((uint64_t)n * m >> 32) + n) >> s);
  }
  constexpr uint32_t mod(uint32_t n) const { return n - div(n) * d; }
};

}  // namespace mk
