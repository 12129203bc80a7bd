// Host check of the slice geometry used by the decode kernels (SliceGeom):
// slice_start and slice_of, evaluated with fp32 estimates and one integer
// correction, against their exact integer definitions,
//   slice_start(s) = floor(C(s) W / C(n)),  slice_of(x) = largest s with slice_start(s) <= x,
// where C(s) counts one unit per earlier slice, or (eight XCDs, n a multiple
// of 8, at least kXcdWeightMinTiles positions per slice) kXcdEvenUnits per
// earlier slice t with (t / 4) even and kXcdOddUnits per one with (t / 4) odd.
// Every slice boundary of several thousand (W, n) pairs is checked, with and
// without XCD weights. Compiled host-only; prints "ok <cases>" or the first
// mismatch and exits nonzero.
#include <stdint.h>
#include <stdio.h>

#include <random>
#include <vector>

#include "neo_internal.h"

static bool check(int64_t W, int64_t n, bool xcd8) {
  const neo::SliceGeom g = neo::make_slice_geom((int32_t)W, (int32_t)n, xcd8);
  const bool weighted = xcd8 && n % 8 == 0 && W >= neo::kXcdWeightMinTiles * n;
  if ((g.weighted != 0) != weighted) {
    printf("weighted flag W=%lld n=%lld\n", (long long)W, (long long)n);
    return false;
  }
  // C(s) by its definition, slice by slice.
  std::vector<int64_t> units(n + 1, 0);
  for (int64_t t = 0; t < n; ++t)
    units[t + 1] = units[t] + (!weighted ? 1 : ((t / 4) % 2 == 0 ? neo::kXcdEvenUnits
                                                                 : neo::kXcdOddUnits));
  std::vector<int64_t> start(n + 1);
  for (int64_t s = 0; s <= n; ++s) {
    start[s] = units[s] * W / units[n];
    if (neo::slice_start((int32_t)s, g) != start[s]) {
      printf("slice_start W=%lld n=%lld s=%lld (weighted %d): %d != %lld\n", (long long)W,
             (long long)n, (long long)s, (int)weighted, neo::slice_start((int32_t)s, g),
             (long long)start[s]);
      return false;
    }
    if (s > 0 && start[s] <= start[s - 1]) {
      printf("empty slice W=%lld n=%lld s=%lld\n", (long long)W, (long long)n, (long long)s);
      return false;
    }
  }
  // Positions around each slice's first and last: slice_of must return s
  // inside [start(s), start(s+1)).
  for (int64_t s = 0; s < n; ++s) {
    const int64_t xs[4] = {start[s], start[s] + 1, start[s + 1] - 2, start[s + 1] - 1};
    for (int64_t x : xs) {
      if (x < start[s] || x >= start[s + 1]) continue;
      const int32_t got = neo::slice_of((int32_t)x, g);
      if (got != s) {
        printf("slice_of W=%lld n=%lld x=%lld (weighted %d): %d != %lld\n", (long long)W,
               (long long)n, (long long)x, (int)weighted, got, (long long)s);
        return false;
      }
    }
  }
  return true;
}

int main() {
  std::mt19937_64 rng(12345);
  long cases = 0, weighted_cases = 0;
  auto run = [&](int64_t W, int64_t n) {
    if (n < 1 || n > NEO_MAX_SLICES || W < n || W > INT32_MAX) return true;
    for (bool xcd8 : {false, true}) {
      ++cases;
      if (xcd8 && n % 8 == 0 && W >= neo::kXcdWeightMinTiles * n) ++weighted_cases;
      if (!check(W, n, xcd8)) return false;
    }
    return true;
  };
  for (int64_t n = 1; n <= 300; ++n)
    for (int64_t W : {n, n + 1, 2 * n - 1, 2 * n, 8 * n + 3, 128 * n - 1, 128 * n, 300 * n + 7,
                      (int64_t)44213, (int64_t)1000003, (int64_t)INT32_MAX})
      if (!run(W, n)) return 1;
  const int64_t big_n[] = {511, 512, 1023, 1024, 1025, 2047, 2048, 3000, 4088, 4095, 4096};
  for (int64_t n : big_n)
    for (int64_t W : {n, n + 1, 2 * n - 1, 2 * n, 3 * n - 1, 8 * n, 8 * n + 7, 128 * n - 1,
                      128 * n, 128 * n + 1, 213 * n + 5, 560 * n + 3, (int64_t)44213,
                      (int64_t)349824, (int64_t)2359296, (int64_t)4589000, (int64_t)16777216,
                      (int64_t)16777217, (int64_t)123456789, (int64_t)INT32_MAX - 1,
                      (int64_t)INT32_MAX})
      if (!run(W, n)) return 1;
  for (int i = 0; i < 2000; ++i) {
    int64_t n = 1 + (int64_t)(rng() % NEO_MAX_SLICES);
    if (i % 2 == 0) n = 8 * (1 + (int64_t)(rng() % (NEO_MAX_SLICES / 8)));
    const int bits = 1 + (int)(rng() % 31);
    const int64_t W =
        n + (int64_t)(rng() % ((uint64_t)1 << bits)) % ((int64_t)INT32_MAX - n + 1);
    if (!run(W, n)) return 1;
  }
  printf("ok %ld (%ld weighted)\n", cases, weighted_cases);
  return 0;
}
