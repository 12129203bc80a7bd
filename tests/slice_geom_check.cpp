// Host check of the slice geometry used by the decode kernels (SliceGeom):
// slice_start and slice_of, evaluated with fp32 estimates and one integer
// correction, against the exact 64-bit integer definitions
//   slice_start(s) = floor(s W / n),  slice_of(x) = largest s with slice_start(s) <= x,
// for every slice of many (W, n). Compiled host-only; prints "ok <cases>" or
// the first mismatch and exits nonzero.
#include <stdint.h>
#include <stdio.h>

#include <random>

#include "neo_internal.h"

static int64_t exact_start(int64_t s, int64_t W, int64_t n) { return s * W / n; }

static bool check(int32_t W, int32_t n) {
  const neo::SliceGeom g = neo::make_slice_geom(W, n);
  for (int32_t s = 0; s <= n; ++s) {
    const int64_t e = exact_start(s, W, n);
    if (neo::slice_start(s, g) != e) {
      printf("slice_start W=%d n=%d s=%d: %d != %lld\n", W, n, s, neo::slice_start(s, g),
             (long long)e);
      return false;
    }
    if (s == n) break;
    // Positions around the slice's first and last: slice_of must return s
    // inside [start(s), start(s+1)).
    const int64_t e1 = exact_start(s + 1, W, n);
    const int64_t xs[4] = {e, e + 1, e1 - 2, e1 - 1};
    for (int64_t x : xs) {
      if (x < e || x >= e1) continue;
      const int32_t got = neo::slice_of((int32_t)x, g);
      if (got != s) {
        printf("slice_of W=%d n=%d x=%lld: %d != %d\n", W, n, (long long)x, got, s);
        return false;
      }
    }
  }
  return true;
}

int main() {
  std::mt19937_64 rng(12345);
  long cases = 0;
  auto run = [&](int64_t W, int64_t n) {
    if (n < 1 || n > NEO_MAX_SLICES || W < n || W > INT32_MAX) return true;
    ++cases;
    return check((int32_t)W, (int32_t)n);
  };
  for (int32_t n = 1; n <= 300; ++n)
    for (int64_t W : {(int64_t)n, (int64_t)n + 1, 2 * (int64_t)n - 1, 2 * (int64_t)n,
                      8 * (int64_t)n + 3, (int64_t)44213, (int64_t)1000003, (int64_t)INT32_MAX})
      if (!run(W, n)) return 1;
  const int64_t big_n[] = {511, 512, 1023, 1024, 1025, 2047, 2048, 3000, 4095, 4096};
  for (int64_t n : big_n)
    for (int64_t W : {n, n + 1, 2 * n - 1, 2 * n, 3 * n - 1, 8 * n, 8 * n + 7, (int64_t)44213,
                      (int64_t)44214, (int64_t)349824, (int64_t)2359296, (int64_t)4589000,
                      (int64_t)16777216, (int64_t)16777217, (int64_t)123456789,
                      (int64_t)INT32_MAX - 1, (int64_t)INT32_MAX})
      if (!run(W, n)) return 1;
  for (int i = 0; i < 3000; ++i) {
    const int64_t n = 1 + (int64_t)(rng() % NEO_MAX_SLICES);
    const int bits = 1 + (int)(rng() % 31);
    const int64_t W = n + (int64_t)(rng() % ((uint64_t)1 << bits)) % ((int64_t)INT32_MAX - n + 1);
    if (!run(W, n)) return 1;
  }
  printf("ok %ld\n", cases);
  return 0;
}
