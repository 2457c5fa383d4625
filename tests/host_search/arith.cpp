// arith.cpp -- test harness: the device's integer ceiling division of the
// processor-sharing evaluator (ceil_div_small in kernels.h, host build)
// against exact 128-bit division, for every rate w in [256, 2^16] (the rates
// round(2^32 / F) of factors F in [2^16, 2^24]) and dividends at and around
// multiples of w up to the largest work 2^46 - 1.  Prints the number of
// mismatches and of cases checked.
#include "../../paper_2607_22242_amd/csrc/kernels.h"

#include <cstdio>

int main() {
  using devmap::ceil_div_small;
  unsigned long long bad = 0, checked = 0;
  const uint64_t amax = (uint64_t(1) << 46) - 1;
  uint64_t seed = 0x9E3779B97F4A7C15ull;
  for (uint32_t w = 256; w <= 65536; ++w) {
    const uint64_t winv = (uint64_t(1) << 48) / w;
    const uint64_t qmax = amax / w;
    uint64_t as[24];
    int n = 0;
    as[n++] = 0;
    as[n++] = 1;
    as[n++] = amax;
    as[n++] = amax - 1;
    as[n++] = qmax * w;
    as[n++] = qmax * w - 1;
    for (int k = 0; k < 6; ++k) {
      seed ^= seed << 13;
      seed ^= seed >> 7;
      seed ^= seed << 17;
      const uint64_t q = seed % (qmax + 1);
      as[n++] = q * w;
      if (q * w > 0) as[n++] = q * w - 1;
      if (q * w + 1 <= amax) as[n++] = q * w + 1;
    }
    for (int i = 0; i < n; ++i) {
      const uint64_t a = as[i];
      const uint64_t want = a / w + (a % w != 0 ? 1 : 0);
      if (ceil_div_small(a, w, winv) != want) ++bad;
      ++checked;
    }
  }
  printf("%llu %llu\n", bad, checked);
  return bad != 0;
}
