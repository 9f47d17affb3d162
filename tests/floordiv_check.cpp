// Host-side check of the exact floor division used by the routing scorer:
// floordiv_exact(a, d, 1/d) must equal a / d (C integer division; both
// operands are non-negative, so truncation is the floor) for every divisor in
// [1, 5000], divisors near 2^31, and dividends at and around multiples of d up
// to 2^50, plus pseudo-random dividends.  Prints the number of mismatches.
#include <cstdio>
#include <cstdint>
#include "common.hpp"

static uint64_t state = 0x9E3779B97F4A7C15ull;
static uint64_t next_rand() {  // splitmix64
  uint64_t z = (state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

static long long bad = 0, checked = 0;
static void check(int64_t a, int32_t d) {
  if (a < 0 || a >= (int64_t(1) << 50)) return;
  const int64_t got = nalar::floordiv_exact(double(a), d, 1.0 / double(d));
  ++checked;
  if (got != a / d) {
    if (bad < 10) std::printf("mismatch a=%lld d=%d got=%lld want=%lld\n", (long long)a, d,
                              (long long)got, (long long)(a / d));
    ++bad;
  }
}

int main() {
  const int64_t top = (int64_t(1) << 50) - 1;
  for (int32_t d = 1; d <= 5000; ++d) {
    for (int64_t a = 0; a < 3 * d; ++a) check(a, d);
    for (int64_t q : {int64_t(1) << 20, int64_t(1) << 30, top / d - 1, top / d}) {
      for (int64_t o = -2; o <= 2; ++o) check(q * d + o, d);
    }
    for (int i = 0; i < 200; ++i) check(int64_t(next_rand() & uint64_t(top)), d);
    for (int i = 0; i < 50; ++i) {
      const int64_t q = int64_t(next_rand() % uint64_t(top / d + 1));
      check(q * d, d); check(q * d - 1, d); check(q * d + d - 1, d);
    }
  }
  for (int32_t d : {2147483647, 2147483646, 1 << 30, 65537, 999983}) {
    for (int i = 0; i < 100000; ++i) check(int64_t(next_rand() & uint64_t(top)), d);
    for (int64_t q = 0; q < 1000; ++q) { check(q * d, d); check(q * d - 1, d); check(q * d + 1, d); }
  }
  // service times as the scorer sees them: est * 1000 with est <= 2^40
  for (int32_t d = 1; d <= 3000; ++d)
    for (int i = 0; i < 100; ++i) check(int64_t(next_rand() % ((uint64_t(1) << 40) + 1)) * 1000, d);
  std::printf("checked %lld mismatches %lld\n", checked, bad);
  return bad == 0 ? 0 : 1;
}
