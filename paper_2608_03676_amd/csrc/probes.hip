// Peak probes of the MI355X units the planner's kernels lean on: HBM read
// bandwidth, unpacked fp32 FMA issue, the v_exp_f32 rate (alone and beside
// FMAs) and LDS read bandwidth.  Measurement helpers for the benchmark, not
// part of the planner; see include/taot_probes.h.
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "taot_probes.h"

namespace {

constexpr int kThreads = 256;
typedef float v4f __attribute__((ext_vector_type(4)));

// Streams `n4` 16-byte words once: each block reads its own contiguous
// chunk of `per_block` words in batches of 8 non-temporal 16-byte loads per
// thread, the next batch in flight while the current one is summed; one
// partial sum per block so the loads are not dead.
__global__ void __launch_bounds__(kThreads) hbm_read_kernel(const v4f* __restrict__ src, int64_t n4,
                                                            int64_t per_block, float* __restrict__ out) {
  constexpr int U = 8;
  const int64_t lo = (int64_t)blockIdx.x * per_block;
  const int64_t hi = lo + per_block < n4 ? lo + per_block : n4;
  v4f acc = {0.f, 0.f, 0.f, 0.f};
  int64_t i = lo + threadIdx.x;
  v4f a[U], b[U];
  const bool full = hi - lo == per_block && per_block % (2 * U * kThreads) == 0;
  if (full) {
#pragma unroll
    for (int u = 0; u < U; ++u) a[u] = __builtin_nontemporal_load(src + i + u * kThreads);
    for (; i + 2 * U * kThreads <= hi; i += 2 * U * kThreads) {
#pragma unroll
      for (int u = 0; u < U; ++u) b[u] = __builtin_nontemporal_load(src + i + (U + u) * kThreads);
#pragma unroll
      for (int u = 0; u < U; ++u) acc += a[u];
      if (i + 3 * U * kThreads <= hi) {
#pragma unroll
        for (int u = 0; u < U; ++u) a[u] = __builtin_nontemporal_load(src + i + (2 * U + u) * kThreads);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) acc += b[u];
    }
  } else {
    for (; i < hi; i += kThreads) acc += __builtin_nontemporal_load(src + i);
  }
  __shared__ float red[kThreads];
  red[threadIdx.x] = (acc.x + acc.y) + (acc.z + acc.w);
  __syncthreads();
  if (threadIdx.x == 0) {
    float s = 0.f;
    for (int t = 0; t < kThreads; ++t) s += red[t];
    out[blockIdx.x] = s;
  }
}

// 8 independent FMA chains per lane, `iters` x 8 FMAs each, in the
// accumulate form a += b * m of the planner's mat-vecs (v_fmac_f32; plus 8
// adds to combine the chains at the end).
__global__ void __launch_bounds__(kThreads) fma_kernel(int32_t iters, float m, float* __restrict__ out) {
  float a[8], b[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    a[k] = (float)(threadIdx.x + k);
    b[k] = 1e-3f * (float)(k + 1);
  }
  for (int32_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
      for (int k = 0; k < 8; ++k) a[k] = __builtin_fmaf(b[k], m, a[k]);
  }
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < 8; ++k) s += a[k];
  out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = s;
}

// 8 independent v_exp_f32 chains per lane, `iters` x 8 exponentials each;
// with `fmas` set, each exponential is joined by one independent FMA chain
// step (to see whether the two issue together).
template <bool FMAS>
__global__ void __launch_bounds__(kThreads) exp_kernel(int32_t iters, float m, float* __restrict__ out) {
  float a[8], b[8], w[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    a[k] = 1e-3f * (float)(threadIdx.x + k);
    b[k] = (float)k;
    w[k] = 1e-3f * (float)(k + 1);
  }
  for (int32_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        a[k] = __builtin_amdgcn_exp2f(-a[k]);  // one v_exp_f32 (negated input); stays in (0, 1]
        if (FMAS) b[k] = __builtin_fmaf(w[k], m, b[k]);
      }
  }
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < 8; ++k) s += a[k] + b[k];
  out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = s;
}

// Each wave reads 16-byte words of a 32 KiB LDS table, consecutive lanes at
// consecutive words (no bank conflicts), `iters` x 8 reads per lane.
__global__ void __launch_bounds__(kThreads) lds_kernel(int32_t iters, float* __restrict__ out) {
  __shared__ float4 tab[2048];
  for (int t = threadIdx.x; t < 2048; t += kThreads) tab[t] = make_float4(t, t + 1, t + 2, t + 3);
  __syncthreads();
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  int idx = threadIdx.x;
  for (int32_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const float4 v = tab[(idx + r * kThreads) & 2047];
      acc.x += v.x;
      acc.y += v.y;
      acc.z += v.z;
      acc.w += v.w;
    }
    idx = (idx + 64) & 2047;
  }
  out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = (acc.x + acc.y) + (acc.z + acc.w);
}

taot_probe_status launched() { return hipGetLastError() == hipSuccess ? 0 : 1; }

}  // namespace

extern "C" {

taot_probe_status taot_probe_hbm_read(const void* src, size_t bytes, int32_t blocks, float* out, void* stream) {
  if (!src || !out || bytes < 16 || blocks <= 0 || (reinterpret_cast<uintptr_t>(src) & 15u)) return 2;
  const int64_t n4 = (int64_t)(bytes / 16);
  const int64_t per_block = (n4 + blocks - 1) / blocks;
  hipLaunchKernelGGL(hbm_read_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, static_cast<hipStream_t>(stream),
                     static_cast<const v4f*>(src), n4, per_block, out);
  return launched();
}

taot_probe_status taot_probe_fma(int32_t blocks, int32_t iters, float* out, void* stream) {
  if (!out || blocks <= 0 || iters <= 0) return 2;
  hipLaunchKernelGGL(fma_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, static_cast<hipStream_t>(stream), iters,
                     0.999f, out);
  return launched();
}

taot_probe_status taot_probe_exp(int32_t blocks, int32_t iters, int32_t with_fma, float* out, void* stream) {
  if (!out || blocks <= 0 || iters <= 0) return 2;
  if (with_fma)
    hipLaunchKernelGGL(exp_kernel<true>, dim3((unsigned)blocks), dim3(kThreads), 0, static_cast<hipStream_t>(stream),
                       iters, 0.999f, out);
  else
    hipLaunchKernelGGL(exp_kernel<false>, dim3((unsigned)blocks), dim3(kThreads), 0,
                       static_cast<hipStream_t>(stream), iters, 0.999f, out);
  return launched();
}

taot_probe_status taot_probe_lds(int32_t blocks, int32_t iters, float* out, void* stream) {
  if (!out || blocks <= 0 || iters <= 0) return 2;
  hipLaunchKernelGGL(lds_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, static_cast<hipStream_t>(stream), iters,
                     out);
  return launched();
}

}  // extern "C"
