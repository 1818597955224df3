// Step 3 of the planner: batched Phase-1 Sinkhorn-Knopp (Sec. A.2).
//
// The paper's iteration is the linear-domain pair u = s~ / (M v),
// v = d / (M^T u) with M = exp(-C / eps), T = diag(u) M diag(v).  In fp32 the
// kernel M underflows for the costs used here (exp(-8 / 0.08)), so the
// iterate is carried in the stabilised form of Schmitzer (2019, "Stabilized
// sparse scaling algorithms for entropy regularized transport problems"):
//     T = diag(u) Kt diag(v),  Kt_ij = exp2(F_i + G_j - C'_ij),  C' = C log2(e) / eps,
// where F, G are absorbed potentials (log2 units) and u, v are scalings kept
// in [2^-20, 2^20].  One half-step is one GEMV-like sweep with one FMA per
// entry; when a scaling leaves its range (or its sum under/overflows) that
// row or column is recomputed exactly in the log domain (max-shifted
// log-sum-exp over the current potentials), absorbed into F or G and its Kt
// entries rebuilt.  In exact arithmetic this is the same iterate as the
// paper's update; the fp32 result agrees with the fp64 definition to
// rounding.
//
// Support.  Supply is zero off the hot set H = {a > 0} and demand is zero off
// the cold set C = {b > 0} (Sec. A.2), so after the first column update every
// potential off H x C is -inf and the iterate lives on the |H| x |C| block.
// The first row update is taken over all R columns (the start v = 1 covers
// every column).
//
// Launches.  sinkhorn_kernel<false> keeps Kt in LDS (one workgroup per problem,
// all iterations fused); problems whose block does not fit are flagged and
// handled by sinkhorn_kernel<true>, which streams Kt through device memory
// (L2-resident at the sizes used here).
#include "common.h"

namespace taot {
namespace {

constexpr int kSkThreads = 256;
constexpr int kSkWaves = kSkThreads / kWave;
constexpr float kLo = 0x1p-20f;
constexpr float kHi = 0x1p20f;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kLdsMaxR = 256;            // beyond this every problem is streamed
constexpr int kVecArrays = 11;           // per-problem vectors of length R in LDS

__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float flog2(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float frcp(float x) { return __builtin_amdgcn_rcpf(x); }

struct SkParams {
  const float* a;
  const float* b;
  int32_t B, R;
  const float* C;
  int64_t C_stride;
  float eps;
  int32_t iters;
  uint32_t flags;
  float* T;
  float* f;
  float* g;
  uint32_t* status;
  int32_t* stream_flag;  // [B] 1 = problem left to the streamed kernel
  float* kt_ws;          // streamed Kt storage, kt_stride floats per problem
  int64_t kt_stride;
  int32_t lds_kt_cap;    // Kt capacity (floats) of the LDS kernel
  int32_t all_streamed;  // every problem goes to the streamed kernel
};

// Block-wide exclusive compaction position of `flag` within a 256-thread chunk.
__device__ __forceinline__ int32_t chunk_compact(bool flag, int32_t* wave_cnt, int32_t& total) {
  const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
  const uint64_t m = __ballot(flag);
  const int32_t lp = __popcll(m & ((1ull << lane) - 1ull));
  if (lane == 0) wave_cnt[wid] = __popcll(m);
  __syncthreads();
  int32_t off = 0, tot = 0;
  for (int w = 0; w < kSkWaves; ++w) {
    const int32_t c = wave_cnt[w];
    off += w < wid ? c : 0;
    tot += c;
  }
  __syncthreads();
  total = tot;
  return off + lp;
}

template <bool STREAM>
__global__ void __launch_bounds__(kSkThreads) sinkhorn_kernel(SkParams p) {
  extern __shared__ float lds[];
  __shared__ int32_t wave_cnt[kSkWaves];
  __shared__ double red_d[2][kSkWaves];
  __shared__ int32_t sh_bad;

  const int64_t pb = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
  const int32_t R = p.R;
  const float* a = p.a + pb * R;
  const float* bd = p.b + pb * R;
  const float* Cb = p.C + pb * p.C_stride;

  if (STREAM && !p.all_streamed && p.stream_flag[pb] == 0) return;  // uniform per block

  int32_t* hidx = reinterpret_cast<int32_t*>(lds);
  int32_t* cidx = hidx + R;
  int32_t* hpos = cidx + R;
  int32_t* cpos = hpos + R;
  float* sA = reinterpret_cast<float*>(cpos + R);
  float* sB = sA + R;
  float* F = sB + R;
  float* G = F + R;
  float* u = G + R;
  float* v = u + R;
  float* cap = v + R;
  float* Kt = cap + R;  // LDS variant only

  // ---- supply/demand: validation, mass, compaction of H and C ----------------
  if (tid == 0) sh_bad = 0;
  __syncthreads();
  double sa = 0.0, sd = 0.0;
  for (int32_t i = tid; i < R; i += kSkThreads) {
    const float ai = a[i], bi = bd[i];
    if (!(ai >= 0.f && ai <= 3.402823466e38f) || !(bi >= 0.f && bi <= 3.402823466e38f)) sh_bad = 1;
    sa += (double)ai;
    sd += (double)bi;
    hpos[i] = -1;
    cpos[i] = -1;
  }
  sa = wave_sum_d(sa);
  sd = wave_sum_d(sd);
  if (lane == 0) { red_d[0][wid] = sa; red_d[1][wid] = sd; }
  __syncthreads();
  double Sa = 0.0, Sd = 0.0;
  for (int w = 0; w < kSkWaves; ++w) { Sa += red_d[0][w]; Sd += red_d[1][w]; }
  double gamma = Sd / (Sa > kEps0 ? Sa : kEps0);
  gamma = gamma < 1.0 ? gamma : 1.0;

  int32_t nh = 0, nc = 0;
  for (int32_t base = 0; base < R; base += kSkThreads) {
    const int32_t i = base + tid;
    const bool in = i < R;
    const float ai = in ? a[i] : 0.f, bi = in ? bd[i] : 0.f;
    int32_t th, tc;
    const int32_t ph = chunk_compact(in && ai > 0.f, wave_cnt, th);
    if (in && ai > 0.f) { hidx[nh + ph] = i; hpos[i] = nh + ph; sA[nh + ph] = (float)(gamma * (double)ai); }
    const int32_t pc = chunk_compact(in && bi > 0.f, wave_cnt, tc);
    if (in && bi > 0.f) { cidx[nc + pc] = i; cpos[i] = nc + pc; sB[nc + pc] = bi; }
    nh += th;
    nc += tc;
  }
  __syncthreads();

  // ---- where the Kt block lives ----------------------------------------------
  const int64_t need = (int64_t)nh * nc;
  const bool degenerate = sh_bad || nh == 0 || nc == 0;
  if (!STREAM) {
    const bool to_stream = !degenerate && (need > p.lds_kt_cap || (p.flags & TAOT_SK_FORCE_STREAM));
    if (tid == 0) p.stream_flag[pb] = to_stream ? 1 : 0;
    if (to_stream) return;
  }
  float* K = STREAM ? p.kt_ws + pb * p.kt_stride : Kt;
  const float kappa = kLog2e / p.eps;  // C' = C * log2(e) / eps

  // ---- first row update over all R columns (g = 0): F_i = log2 s~_i - LSE2_j(-C'_ij)
  if (!degenerate) {
    for (int32_t ii = wid; ii < nh; ii += kSkWaves) {
      const float* crow = Cb + (int64_t)hidx[ii] * R;
      float mx = -INFINITY;
      bool badc = false;
      for (int32_t j = lane; j < R; j += kWave) {
        const float c = crow[j];
        badc |= !(c == c) || c == INFINITY || c == -INFINITY;
        mx = fmaxf(mx, -c * kappa);
      }
      if (badc) sh_bad = 1;
      mx = wave_max(mx);
      float s = 0.f;
      for (int32_t j = lane; j < R; j += kWave) s += fexp2(-crow[j] * kappa - mx);
      s = wave_sum(s);
      if (lane == 0) { F[ii] = flog2(sA[ii]) - (mx + flog2(s)); u[ii] = 1.f; }
    }
    for (int32_t jj = tid; jj < nc; jj += kSkThreads) { G[jj] = 0.f; v[jj] = 1.f; }
  }
  __syncthreads();

  uint32_t st = 0;
  if (sh_bad) st = TAOT_ST_BAD_INPUT;
  else if (nh == 0 || nc == 0) st = TAOT_ST_ZERO_MASS;
  if (st) {
    if (p.T)
      for (int64_t q = tid; q < (int64_t)R * R; q += kSkThreads) p.T[pb * R * R + q] = 0.f;
    for (int32_t i = tid; i < R; i += kSkThreads) {
      if (p.f) p.f[pb * R + i] = -INFINITY;
      if (p.g) p.g[pb * R + i] = -INFINITY;
    }
    if (tid == 0 && p.status) p.status[pb] = st;
    return;
  }

  // ---- build Kt = exp2(F_i + G_j - C'_ij) on H x C ----------------------------
  for (int64_t q = tid; q < need; q += kSkThreads) {
    const int32_t ii = (int32_t)(q / nc), jj = (int32_t)(q % nc);
    const float c = Cb[(int64_t)hidx[ii] * R + cidx[jj]];
    K[q] = fexp2((F[ii] + G[jj]) - c * kappa);
  }
  __syncthreads();

  for (int32_t it = 1; it <= p.iters; ++it) {
    if (it > 1) {
      // ---- row update: u_i = s~_i / sum_j Kt_ij v_j  (one wave per row) -------
      for (int32_t ii = wid; ii < nh; ii += kSkWaves) {
        const float* krow = K + (int64_t)ii * nc;
        float y = 0.f;
        for (int32_t jj = lane; jj < nc; jj += kWave) y = __builtin_fmaf(krow[jj], v[jj], y);
        // lanes may differ in the last bit of a butterfly sum: use lane 0's value
        y = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(wave_sum(y))));
        const float un = sA[ii] * frcp(y);
        if (un >= kLo && un <= kHi) {
          if (lane == 0) u[ii] = un;
        } else {
          // exact log-domain update of row ii, absorbed into F
          const float* crow = Cb + (int64_t)hidx[ii] * R;
          float mx = -INFINITY;
          for (int32_t jj = lane; jj < nc; jj += kWave)
            mx = fmaxf(mx, (G[jj] + flog2(v[jj])) - crow[cidx[jj]] * kappa);
          mx = wave_max(mx);
          float s = 0.f;
          for (int32_t jj = lane; jj < nc; jj += kWave)
            s += fexp2(((G[jj] + flog2(v[jj])) - crow[cidx[jj]] * kappa) - mx);
          s = wave_sum(s);
          const float fi = flog2(sA[ii]) - (mx + flog2(s));
          for (int32_t jj = lane; jj < nc; jj += kWave)
            K[(int64_t)ii * nc + jj] = fexp2((fi + G[jj]) - crow[cidx[jj]] * kappa);
          if (lane == 0) { F[ii] = fi; u[ii] = 1.f; }
        }
      }
      __syncthreads();
    }
    // ---- column update: v_j = d_j / sum_i u_i Kt_ij  (one thread per column) ---
    for (int32_t jj = tid; jj < nc; jj += kSkThreads) {
      float x = 0.f;
      for (int32_t ii = 0; ii < nh; ++ii) x = __builtin_fmaf(u[ii], K[(int64_t)ii * nc + jj], x);
      const float vn = sB[jj] * frcp(x);
      if (vn >= kLo && vn <= kHi) {
        v[jj] = vn;
      } else {
        // exact log-domain update of column jj, absorbed into G
        const int32_t j = cidx[jj];
        float mx = -INFINITY;
        for (int32_t ii = 0; ii < nh; ++ii)
          mx = fmaxf(mx, (F[ii] + flog2(u[ii])) - Cb[(int64_t)hidx[ii] * R + j] * kappa);
        float s = 0.f;
        for (int32_t ii = 0; ii < nh; ++ii)
          s += fexp2(((F[ii] + flog2(u[ii])) - Cb[(int64_t)hidx[ii] * R + j] * kappa) - mx);
        const float gj = flog2(sB[jj]) - (mx + flog2(s));
        for (int32_t ii = 0; ii < nh; ++ii)
          K[(int64_t)ii * nc + jj] = fexp2((F[ii] + gj) - Cb[(int64_t)hidx[ii] * R + j] * kappa);
        G[jj] = gj;
        v[jj] = 1.f;
      }
    }
    __syncthreads();
  }

  // ---- plan, column cap, outputs -----------------------------------------------
  const bool colcap = !(p.flags & TAOT_SK_NO_COLCAP);
  for (int32_t jj = tid; jj < nc; jj += kSkThreads) {
    float c = 0.f;
    if (colcap)
      for (int32_t ii = 0; ii < nh; ++ii) c += u[ii] * K[(int64_t)ii * nc + jj] * v[jj];
    const float fac = colcap ? fminf(1.f, sB[jj] / (c + 1e-12f)) : 1.f;
    cap[jj] = v[jj] * fac;
  }
  __syncthreads();
  if (p.T) {
    float* Tb = p.T + pb * R * R;
    for (int32_t i = 0; i < R; ++i) {
      const int32_t ii = hpos[i];
      for (int32_t j = tid; j < R; j += kSkThreads) {
        const int32_t jj = cpos[j];
        Tb[(int64_t)i * R + j] = (ii >= 0 && jj >= 0) ? u[ii] * K[(int64_t)ii * nc + jj] * cap[jj] : 0.f;
      }
    }
  }
  const float to_nat = p.eps * kLn2;  // log2 units -> eps * ln
  for (int32_t i = tid; i < R; i += kSkThreads) {
    const int32_t ii = hpos[i], jj = cpos[i];
    if (p.f) p.f[pb * R + i] = ii >= 0 ? (F[ii] + flog2(u[ii])) * to_nat : -INFINITY;
    if (p.g) p.g[pb * R + i] = jj >= 0 ? (G[jj] + flog2(v[jj])) * to_nat : -INFINITY;
  }
  if (tid == 0 && p.status) p.status[pb] = STREAM ? TAOT_ST_STREAMED : 0u;
}

// Largest nh * nc over disjoint supports of R ranks (nh + nc <= R).
int64_t max_block(int32_t R) { return (int64_t)(R / 2) * (R - R / 2); }

struct SkWs {
  int32_t* flag;
  float* kt;
  int64_t kt_stride;
  size_t bytes;
};

SkWs carve(void* ws, int32_t B, int32_t R) {
  Carver c{static_cast<char*>(ws)};
  SkWs w;
  w.flag = c.take<int32_t>((size_t)B);
  w.kt_stride = round_up((int64_t)R * R, 64);
  w.kt = c.take<float>((size_t)B * w.kt_stride);
  w.bytes = c.off;
  return w;
}

}  // namespace

size_t sinkhorn_ws(int32_t B, int32_t R) { return carve(nullptr, B, R).bytes; }

taot_status launch_sinkhorn(const float* a, const float* b, int32_t B, int32_t R, const float* C,
                            int64_t C_stride, float eps, int32_t iters, uint32_t flags, float* T,
                            float* f, float* g, uint32_t* status, void* ws, hipStream_t stream) {
  if (B == 0) return TAOT_OK;
  SkWs w = carve(ws, B, R);
  SkParams p{a, b, B, R, C, C_stride, eps, iters, flags, T, f, g, status, w.flag, w.kt, w.kt_stride, 0, 0};
  const size_t vec_bytes = (size_t)kVecArrays * R * sizeof(float);
  const bool lds_path = R <= kLdsMaxR;
  if (lds_path) {
    p.lds_kt_cap = (int32_t)max_block(R);
    const size_t lds = vec_bytes + (size_t)p.lds_kt_cap * sizeof(float);
    if (lds > 65536 && hipFuncSetAttribute((const void*)sinkhorn_kernel<false>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)lds) != hipSuccess)
      return TAOT_ERR_LAUNCH;
    hipLaunchKernelGGL(sinkhorn_kernel<false>, dim3((unsigned)B), dim3(kSkThreads), lds, stream, p);
    if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  } else {
    p.all_streamed = 1;
  }
  if (vec_bytes > 65536 && hipFuncSetAttribute((const void*)sinkhorn_kernel<true>,
                                               hipFuncAttributeMaxDynamicSharedMemorySize,
                                               (int)vec_bytes) != hipSuccess)
    return TAOT_ERR_LAUNCH;
  hipLaunchKernelGGL(sinkhorn_kernel<true>, dim3((unsigned)B), dim3(kSkThreads), vec_bytes, stream, p);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  return TAOT_OK;
}

}  // namespace taot
