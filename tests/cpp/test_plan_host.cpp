// Host-only checks of the plan helpers (built with g++, no HIP): the
// multiply-shift division against hardware division, and kept-row counts
// against a direct enumeration.
#include <cstdio>
#include <cstdlib>
#include <cstdint>
#include <random>

#include "plan.h"

static int fails = 0;
#define CHECK(c) do { if (!(c)) { std::printf("FAIL %s:%d %s\n", __FILE__, __LINE__, #c); if (++fails > 20) std::exit(1); } } while (0)

int main() {
  std::mt19937_64 rng(12345);
  const uint32_t lim = 0x7fffffffu;
  // divisors: small, powers of two and neighbours, random, largest
  std::vector<uint32_t> ds;
  for (uint32_t d = 1; d < 4096; ++d) ds.push_back(d);
  for (int b = 1; b < 31; ++b) { ds.push_back(1u << b); ds.push_back((1u << b) - 1); ds.push_back((1u << b) + 1); }
  for (int i = 0; i < 2000; ++i) ds.push_back(1 + static_cast<uint32_t>(rng() % lim));
  ds.push_back(lim);
  for (uint32_t d : ds) {
    const da::FastDiv f = da::make_fastdiv(d);
    CHECK(f.d == d);
    const uint32_t ns[] = {0u, 1u, d - 1, d, d + 1 > d ? d + 1 : d, lim, lim - 1, 2 * d < lim ? 2 * d - 1 : 7u};
    for (uint32_t n : ns) if (n <= lim) CHECK(f.div(n) == n / d);
    for (int i = 0; i < 200; ++i) {
      const uint32_t n = static_cast<uint32_t>(rng() % (uint64_t(lim) + 1));
      CHECK(f.div(n) == n / d);
    }
  }
  // kept rows of a segment: count of t >= 0 with s + t r < len
  for (int64_t len = 0; len < 60; ++len)
    for (int64_t r = 1; r < 20; ++r)
      for (int64_t s = 0; s < 25; ++s) {
        int64_t c = 0;
        for (int64_t p = s; p < len; p += r) ++c;
        CHECK(da::kept_rows(len, s, r) == c);
      }
  std::printf(fails ? "FAILED %d\n" : "OK\n", fails);
  return fails ? 1 : 0;
}
