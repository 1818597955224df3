// Internal declarations shared by the libtaot translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "taot.h"

namespace taot {

constexpr int kWave = 64;
constexpr double kEps0 = 1e-12;

__host__ __device__ constexpr int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// ---- workspace carving (host) ---------------------------------------------
struct Carver {
  char* base;
  size_t off = 0;
  template <typename T>
  __host__ __device__ T* take(size_t count) {
    off = (size_t)round_up((int64_t)off, 256);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
};

// ---- device helpers ---------------------------------------------------------
// Sum over the 64 lanes of a wave with a fixed butterfly order (deterministic).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ int64_t wave_max_i64(int64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    int64_t w = __shfl_xor(v, o, kWave);
    v = w > v ? w : v;
  }
  return v;
}

// Order-preserving map of a double onto uint64 (for max-reductions by atomics).
__device__ __forceinline__ uint64_t ordered_key(double x) {
  uint64_t u = (uint64_t)__double_as_longlong(x);
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// ---- launchers (one per translation unit) -----------------------------------
taot_status launch_plan_loads(const int32_t* ids, int32_t B, int32_t R, int64_t N, int32_t E,
                              const int32_t* home, int32_t* n, int64_t* load_e, int64_t* load_r,
                              int64_t* excess, int64_t* spare, int64_t* spill, float* supply,
                              float* demand, double* rho, double* alpha, int64_t* bad_ids,
                              int32_t* hot_idx, int32_t* cold_idx, int32_t* hot_cnt, int32_t* cold_cnt,
                              uint32_t* status, void* ws, hipStream_t stream);
size_t plan_loads_ws(int32_t B, int32_t R, int32_t E);
size_t plan_loads_scratch_limit();
void* plan_loads_scratch();

taot_status launch_sinkhorn(const float* a, const float* b, int32_t B, int32_t R, const float* C,
                            int64_t C_stride, float eps, int32_t iters, uint32_t flags, float* T,
                            float* f, float* g, uint32_t* status, void* ws, hipStream_t stream);
size_t sinkhorn_ws(int32_t B, int32_t R);

taot_status launch_schedule(const int32_t* n, const int64_t* spill, const int64_t* spare,
                            const int64_t* excess, const double* alpha, const int32_t* home,
                            const float* T, const double* Bpref, const double* Bauct, int32_t B,
                            int32_t R, int32_t E, int32_t K, double price_step, int64_t t_max,
                            uint32_t flags, int32_t* slot_expert, int64_t* slot_amount, int32_t* X,
                            int64_t* unfilled, int32_t* rounds_used, uint32_t* status, void* ws,
                            hipStream_t stream);
size_t schedule_ws(int32_t B, int32_t R, int32_t E, int32_t K);

}  // namespace taot
