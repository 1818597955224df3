/* Host twin of the seeded routing-id generator; the definition is stated in
 * gen_ids.h.  Input generation only. */
#include "gen_ids.h"

#include <stddef.h>

uint64_t gen_splitmix64_at(uint64_t seed, uint64_t i) {
  uint64_t z = seed + (i + 1u) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

static int32_t lookup(const uint64_t* thr, int32_t E, uint32_t u) {
  int32_t lo = 0, hi = E - 1; /* answer in [lo, hi]; thr[E-1] > u always */
  while (lo < hi) {
    int32_t mid = lo + (hi - lo) / 2;
    if ((uint64_t)u < thr[mid]) hi = mid; else lo = mid + 1;
  }
  return lo;
}

int gen_ids_host(const uint64_t* thr, int32_t E, uint64_t seed, int32_t R, int64_t T,
                 int32_t k, int32_t r0, int32_t r1, int32_t* out) {
  if (!thr || !out || E <= 0 || R <= 0 || T < 0 || k <= 0 || k > GEN_MAX_K || k > E ||
      r0 < 0 || r1 > R || r0 > r1 || thr[E - 1] != (1ull << 32))
    return -1;
#pragma omp parallel for schedule(static)
  for (int64_t row = 0; row < (int64_t)(r1 - r0) * T; ++row) {
    int64_t r = r0 + row / T, t = row % T;
    int32_t chosen[GEN_MAX_K];
    for (int32_t d = 0; d < k; ++d) {
      uint64_t base = ((((uint64_t)r * (uint64_t)T + (uint64_t)t) * (uint64_t)k + (uint64_t)d)
                       << GEN_ATTEMPT_BITS);
      int32_t e = -1;
      for (uint32_t a = 0; a < (1u << GEN_ATTEMPT_BITS) - 1u; ++a) {
        uint32_t u = (uint32_t)(gen_splitmix64_at(seed, base + a) >> 32);
        int32_t c = lookup(thr, E, u);
        int dup = 0;
        for (int32_t q = 0; q < d; ++q) dup |= (chosen[q] == c);
        if (!dup) { e = c; break; }
      }
      if (e < 0) { /* fallback: smallest unused id */
        for (int32_t c = 0; c < E && e < 0; ++c) {
          int dup = 0;
          for (int32_t q = 0; q < d; ++q) dup |= (chosen[q] == c);
          if (!dup) e = c;
        }
      }
      chosen[d] = e;
      out[row * k + d] = e;
    }
  }
  return 0;
}
