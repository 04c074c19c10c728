// Host check of the multiply-shift division used by the element-wise kernels:
// FastDiv(d).div(n) / .mod(n) against n / d and n % d for every divisor class
// (1, powers of two and their neighbours, small primes, large and maximal
// divisors) on boundary and pseudo-random numerators.  Prints the number of
// mismatches and exits non-zero on any.
#include <cstdint>
#include <cstdio>
#include <vector>

#include "fastdiv.hpp"

static uint64_t state = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32() {   // xorshift64*
  state ^= state >> 12;
  state ^= state << 25;
  state ^= state >> 27;
  return (uint32_t)((state * 0x2545F4914F6CDD1Dull) >> 32);
}

int main() {
  std::vector<uint32_t> ds;
  for (uint32_t d = 1; d <= 4096; ++d) ds.push_back(d);
  for (int s = 12; s < 32; ++s) {
    const uint32_t p = 1u << s;
    ds.push_back(p - 1);
    ds.push_back(p);
    ds.push_back(p + 1);
  }
  const uint32_t extra[] = {3136, 50176, 14336, 2048 * 2048u, 0x7FFFFFFFu, 0x80000001u,
                            0xFFFFFFFEu, 0xFFFFFFFFu, 1000000007u, 65521u};
  for (uint32_t d : extra) ds.push_back(d);
  for (int i = 0; i < 2000; ++i) ds.push_back(next_u32() | 1u);
  long bad = 0, checked = 0;
  for (uint32_t d : ds) {
    const mk::FastDiv f(d);
    std::vector<uint32_t> ns = {0u, 1u, d - 1, d, d + 1, 2 * d - 1, 2 * d, 0xFFFFFFFFu,
                                0xFFFFFFFEu, 0x80000000u, 0x7FFFFFFFu};
    const uint32_t qmax = 0xFFFFFFFFu / d;
    for (uint32_t q : {qmax, qmax - 1, qmax / 2}) {
      ns.push_back(q * d);
      ns.push_back(q * d + (d - 1));
      if (q) ns.push_back(q * d - 1);
    }
    for (int i = 0; i < 200; ++i) ns.push_back(next_u32());
    for (uint32_t n : ns) {
      ++checked;
      if (f.div(n) != n / d || f.mod(n) != n % d) {
        if (bad < 10) std::printf("mismatch d=%u n=%u: %u vs %u\n", d, n, f.div(n), n / d);
        ++bad;
      }
    }
  }
  std::printf("checked %ld, mismatches %ld\n", checked, bad);
  return bad != 0;
}
