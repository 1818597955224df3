// Device twin of the seeded routing-id generator; the definition is stated in
// gen_ids.h and must match gen_ids.c bit for bit.  Input generation only.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gen_ids.h"

namespace {

constexpr int kThreads = 256;
constexpr int kTokensPerThread = 4;

__device__ __forceinline__ uint64_t splitmix64_at(uint64_t seed, uint64_t i) {
  uint64_t z = seed + (i + 1u) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ int32_t lookup(const uint64_t* thr, int32_t E, uint32_t u) {
  int32_t lo = 0, hi = E - 1;
  while (lo < hi) {
    int32_t mid = lo + (hi - lo) / 2;
    if ((uint64_t)u < thr[mid]) hi = mid; else lo = mid + 1;
  }
  return lo;
}

// One block covers kThreads*kTokensPerThread consecutive tokens of one
// (problem, source rank) row.  Grid: B * R * chunks blocks (1-D).
__global__ void __launch_bounds__(kThreads)
gen_ids_kernel(const uint64_t* __restrict__ thr_all, const uint64_t* __restrict__ seeds, int32_t B,
               int32_t E, int32_t R, int64_t T, int32_t k, int64_t chunks, int32_t* __restrict__ out) {
  extern __shared__ uint64_t thr[];
  const int64_t blk = blockIdx.x;
  const int64_t chunk = blk % chunks;
  const int64_t br = blk / chunks;
  const int32_t r = (int32_t)(br % R);
  const int32_t b = (int32_t)(br / R);
  if (b >= B) return;  // uniform per block
  for (int32_t e = threadIdx.x; e < E; e += kThreads) thr[e] = thr_all[(int64_t)b * E + e];
  __syncthreads();
  const uint64_t seed = seeds[b];
  for (int q = 0; q < kTokensPerThread; ++q) {
    const int64_t t = chunk * (kThreads * kTokensPerThread) + q * kThreads + threadIdx.x;
    if (t >= T) break;
    int32_t chosen[GEN_MAX_K];
    int32_t* dst = out + (((int64_t)b * R + r) * T + t) * k;
    for (int32_t d = 0; d < k; ++d) {
      const uint64_t base =
          ((((uint64_t)r * (uint64_t)T + (uint64_t)t) * (uint64_t)k + (uint64_t)d) << GEN_ATTEMPT_BITS);
      int32_t e = -1;
      for (uint32_t a = 0; a < (1u << GEN_ATTEMPT_BITS) - 1u; ++a) {
        const uint32_t u = (uint32_t)(splitmix64_at(seed, base + a) >> 32);
        const int32_t c = lookup(thr, E, u);
        bool dup = false;
        for (int32_t p = 0; p < d; ++p) dup |= (chosen[p] == c);
        if (!dup) { e = c; break; }
      }
      if (e < 0) {
        for (int32_t c = 0; c < E && e < 0; ++c) {
          bool dup = false;
          for (int32_t p = 0; p < d; ++p) dup |= (chosen[p] == c);
          if (!dup) e = c;
        }
      }
      chosen[d] = e;
      dst[d] = e;
    }
  }
}

}  // namespace

extern "C" {

// Fills ids[B][R][T][k] on `stream`.  thr_all [B][E] and seeds [B] are device
// arrays.  Returns 0, or -1 on invalid arguments / launch failure.
int gen_ids_device(const uint64_t* thr_all, const uint64_t* seeds, int32_t B, int32_t E, int32_t R,
                   int64_t T, int32_t k, int32_t* ids, hipStream_t stream) {
  if (!thr_all || !seeds || !ids || B <= 0 || E <= 0 || E > 8192 || R <= 0 || T <= 0 || k <= 0 ||
      k > GEN_MAX_K || k > E)
    return -1;
  const int64_t per_block = (int64_t)kThreads * kTokensPerThread;
  const int64_t chunks = (T + per_block - 1) / per_block;
  const int64_t blocks = (int64_t)B * R * chunks;
  if (blocks > 0x7fffffffLL) return -1;
  hipLaunchKernelGGL(gen_ids_kernel, dim3((unsigned)blocks), dim3(kThreads), (size_t)E * sizeof(uint64_t),
                     stream, thr_all, seeds, B, E, R, T, k, chunks, ids);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}
