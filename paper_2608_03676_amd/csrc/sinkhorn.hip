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
#include <mutex>

#include "common.h"

namespace taot {
namespace {

constexpr int kSkThreads = 256;
constexpr int kSkWaves = kSkThreads / kWave;
constexpr int kSkStreamThreads = 1024;  // threads per problem of the streamed kernel
constexpr float kLo = 0x1p-20f;
constexpr float kHi = 0x1p20f;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kLdsMaxR = 256;            // beyond this every problem is streamed
constexpr int kVecArrays = 11;           // per-problem vectors of length R in LDS

__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float flog2(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float frcp(float x) { return __builtin_amdgcn_rcpf(x); }

// Register-resident one-wave path: the |H| x |C| block lives on one wave, CPL
// columns per lane (|C| <= 64*CPL) and 8*C8 rows (|H| <= 8*C8).  Class 0 is
// every other problem (degenerate, larger, or the path switched off).
__host__ __device__ constexpr int cpl_index(int cpl) { return cpl == 1 ? 0 : cpl == 2 ? 1 : 2; }
__host__ __device__ constexpr int wave_class(int cpl, int c8) { return 1 + cpl_index(cpl) * 8 + (c8 - 1); }
__device__ __forceinline__ int classify(int32_t nh, int32_t nc, uint32_t flags) {
  if (nh <= 0 || nc <= 0 || nh > 64 || nc > 256) return 0;
  if (flags & (TAOT_SK_FORCE_STREAM | TAOT_SK_NO_REGISTER)) return 0;
  const int cpl = nc <= 64 ? 1 : nc <= 128 ? 2 : 4;
  return wave_class(cpl, (nh + 7) / 8);
}

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

// Block-wide exclusive compaction position of `flag` within an NT-thread chunk.
template <int NT = kSkThreads>
__device__ __forceinline__ int32_t chunk_compact(bool flag, int32_t* wave_cnt, int32_t& total) {
  const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
  const uint64_t m = __ballot(flag);
  const int32_t lp = __popcll(m & ((1ull << lane) - 1ull));
  if (lane == 0) wave_cnt[wid] = __popcll(m);
  __syncthreads();
  int32_t off = 0, tot = 0;
  for (int w = 0; w < NT / kWave; ++w) {
    const int32_t c = wave_cnt[w];
    off += w < wid ? c : 0;
    tot += c;
  }
  __syncthreads();
  total = tot;
  return off + lp;
}

// NT threads per problem: 256 for the LDS variant (several problems per
// compute unit), 1024 for the streamed one (few, large problems).
template <bool STREAM, int NT>
__global__ void __launch_bounds__(NT) sinkhorn_kernel(SkParams p) {
  constexpr int NW = NT / kWave;
  extern __shared__ float lds[];
  __shared__ int32_t wave_cnt[NW];
  __shared__ double red_d[2][NW];
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
  for (int32_t i = tid; i < R; i += NT) {
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
  for (int w = 0; w < NW; ++w) { Sa += red_d[0][w]; Sd += red_d[1][w]; }
  double gamma = Sd / (Sa > kEps0 ? Sa : kEps0);
  gamma = gamma < 1.0 ? gamma : 1.0;

  int32_t nh = 0, nc = 0;
  for (int32_t base = 0; base < R; base += NT) {
    const int32_t i = base + tid;
    const bool in = i < R;
    const float ai = in ? a[i] : 0.f, bi = in ? bd[i] : 0.f;
    int32_t th, tc;
    const int32_t ph = chunk_compact<NT>(in && ai > 0.f, wave_cnt, th);
    if (in && ai > 0.f) { hidx[nh + ph] = i; hpos[i] = nh + ph; sA[nh + ph] = (float)(gamma * (double)ai); }
    const int32_t pc = chunk_compact<NT>(in && bi > 0.f, wave_cnt, tc);
    if (in && bi > 0.f) { cidx[nc + pc] = i; cpos[i] = nc + pc; sB[nc + pc] = bi; }
    nh += th;
    nc += tc;
  }
  __syncthreads();

  // ---- where the Kt block lives ----------------------------------------------
  const int64_t need = (int64_t)nh * nc;
  const bool degenerate = sh_bad || nh == 0 || nc == 0;
  if (!degenerate && classify(nh, nc, p.flags) != 0) {  // the register path owns it
    if (!STREAM && tid == 0) p.stream_flag[pb] = 0;
    return;
  }
  if (!STREAM) {
    const bool to_stream = !degenerate && (need > p.lds_kt_cap || (p.flags & TAOT_SK_FORCE_STREAM));
    if (tid == 0) p.stream_flag[pb] = to_stream ? 1 : 0;
    if (to_stream) return;
  }
  float* K = STREAM ? p.kt_ws + pb * p.kt_stride : Kt;
  const float kappa = kLog2e / p.eps;  // C' = C * log2(e) / eps

  // ---- first row update over all R columns (g = 0): F_i = log2 s~_i - LSE2_j(-C'_ij)
  if (!degenerate) {
    for (int32_t ii = wid; ii < nh; ii += NW) {
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
    for (int32_t jj = tid; jj < nc; jj += NT) { G[jj] = 0.f; v[jj] = 1.f; }
  }
  __syncthreads();

  uint32_t st = 0;
  if (sh_bad) st = TAOT_ST_BAD_INPUT;
  else if (nh == 0 || nc == 0) st = TAOT_ST_ZERO_MASS;
  if (st) {
    if (p.T)
      for (int64_t q = tid; q < (int64_t)R * R; q += NT) p.T[pb * R * R + q] = 0.f;
    for (int32_t i = tid; i < R; i += NT) {
      if (p.f) p.f[pb * R + i] = -INFINITY;
      if (p.g) p.g[pb * R + i] = -INFINITY;
    }
    if (tid == 0 && p.status) p.status[pb] = st;
    return;
  }

  // ---- build Kt = exp2(F_i + G_j - C'_ij) on H x C ----------------------------
  for (int64_t q = tid; q < need; q += NT) {
    const int32_t ii = (int32_t)(q / nc), jj = (int32_t)(q % nc);
    const float c = Cb[(int64_t)hidx[ii] * R + cidx[jj]];
    K[q] = fexp2((F[ii] + G[jj]) - c * kappa);
  }
  __syncthreads();

  for (int32_t it = 1; it <= p.iters; ++it) {
    if (it > 1) {
      // ---- row update: u_i = s~_i / sum_j Kt_ij v_j  (one wave per row) -------
      for (int32_t ii = wid; ii < nh; ii += NW) {
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
    for (int32_t jj = tid; jj < nc; jj += NT) {
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
  for (int32_t jj = tid; jj < nc; jj += NT) {
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
      for (int32_t j = tid; j < R; j += NT) {
        const int32_t jj = cpos[j];
        Tb[(int64_t)i * R + j] = (ii >= 0 && jj >= 0) ? u[ii] * K[(int64_t)ii * nc + jj] * cap[jj] : 0.f;
      }
    }
  }
  const float to_nat = p.eps * kLn2;  // log2 units -> eps * ln
  for (int32_t i = tid; i < R; i += NT) {
    const int32_t ii = hpos[i], jj = cpos[i];
    if (p.f) p.f[pb * R + i] = ii >= 0 ? (F[ii] + flog2(u[ii])) * to_nat : -INFINITY;
    if (p.g) p.g[pb * R + i] = jj >= 0 ? (G[jj] + flog2(v[jj])) * to_nat : -INFINITY;
  }
  if (tid == 0 && p.status) p.status[pb] = STREAM ? TAOT_ST_STREAMED : 0u;
}

// ---------------------------------------------------------------------------
// Register-resident path: one 64-lane wave per problem, no barriers between
// half-steps.  Lane l owns compact columns l, l+64, ... (CPL of them) and holds
// Kt[i][c] for all 8*C8 rows: in VGPRs for the first 8*RC rows, in a per-wave
// LDS tile for the rest (only when CPL = 4 and |H| > 48, which keeps the
// kernel at <= 256 registers and two waves per SIMD).
//   column half-step: x_c = sum_i u_i Kt_ic  (u_i broadcast with v_readlane)
//   row half-step:    p_i = sum_c Kt_ic v_c per lane, then a transposed
//                     butterfly reduce-scatter over the 64 lanes (8 rows at a
//                     time: permlane32/16 swaps, then DPP) leaves the total of
//                     row 8q + (l >> 3) in lane l.
// An out-of-range scaling triggers the exact log-domain update of all rows
// (or all columns) with Kt rebuilt from the new potentials.

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  // every lane has a source lane for the patterns used here, so bound_ctrl
  // changes nothing but lets the move fold into the add
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, true));
}
__device__ __forceinline__ void swap32(float& lo, float& hi) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(lo), __float_as_uint(hi), false, false);
  lo = __uint_as_float(r[0]);
  hi = __uint_as_float(r[1]);
}
__device__ __forceinline__ void swap16(float& lo, float& hi) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(lo), __float_as_uint(hi), false, false);
  lo = __uint_as_float(r[0]);
  hi = __uint_as_float(r[1]);
}
__device__ __forceinline__ float bcast(float x, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), lane));
}
__device__ __forceinline__ float first_lane(float x) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(x)));
}

// Sums 8 per-lane values over the wave; lane l ends with the total of value
// (l >> 3).  Halving steps pair lanes l ^ 32 (permlane32 swap), l ^ 16
// (permlane16 swap) and l <-> 15 - l (row_mirror); the last three steps add
// over l <-> l ^ 7 (row_half_mirror), l ^ 2 and l ^ 1 (quad_perm).
__device__ __forceinline__ float reduce8(float (&p)[8], int lane) {
#pragma unroll
  for (int k = 0; k < 4; ++k) { swap32(p[k], p[k + 4]); p[k] = p[k] + p[k + 4]; }
#pragma unroll
  for (int k = 0; k < 2; ++k) { swap16(p[k], p[k + 2]); p[k] = p[k] + p[k + 2]; }
  const bool b3 = lane & 8;
  const float keep = b3 ? p[1] : p[0];
  const float send = b3 ? p[0] : p[1];
  float y = keep + dpp<0x140>(send);  // row_mirror
  y = y + dpp<0x141>(y);              // row_half_mirror
  y = y + dpp<0x4E>(y);               // quad_perm [2,3,0,1]
  y = y + dpp<0xB1>(y);               // quad_perm [1,0,3,2]
  return y;
}

// Iterations and outputs for one problem of class (CPL, C8); the caller has
// filled the LDS vectors and the first-update potentials Fl.
template <int CPL, int C8>
__device__ __forceinline__ void wave_solve(const SkParams& p, int64_t pb, int32_t nh, int32_t nc,
                                           const int32_t* cpos, const int32_t* hpos, const int32_t* cidx,
                                           const int32_t* hidx, const float* sAl, float* Fl, float* ul,
                                           float kappa) {
  constexpr int MAXH = 8 * C8;
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t R = p.R;
  const float* bd = p.b + pb * R;
  const float* Cb = p.C + pb * p.C_stride;

  float K[MAXH][CPL];
  // row i (static after unrolling) of the lane's columns
  auto kget = [&](int i, int c) -> float { return K[i][c]; };
  auto kset = [&](int i, int c, float val) { K[i][c] = val; };

  // per-lane column state; the column ids and validity are recomputed from
  // LDS / the lane index where needed to keep the kernel within 256 VGPRs
#define CV(c) (lane + kWave * (c) < nc)
#define CJ(c) (CV(c) ? cidx[lane + kWave * (c)] : 0)
  // xb / yb are 1 for padding columns / rows and 0 otherwise: added to the
  // sums of zero padding they keep the scalings finite (0) without selects,
  // and added to the scalings they keep padding inside the range check
  float sB[CPL], G[CPL], v[CPL], xb[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    sB[c] = CV(c) ? bd[CJ(c)] : 0.f;
    G[c] = 0.f;
    v[c] = CV(c) ? 1.f : 0.f;
    xb[c] = CV(c) ? 0.f : 1.f;
  }
  // row-owned values: lane l carries row 8q + (l >> 3) of chunk q
#define RV(q) (8 * (q) + (lane >> 3) < nh)
  float uq[C8], yb[C8];
#pragma unroll
  for (int q = 0; q < C8; ++q) {
    uq[q] = RV(q) ? 1.f : 0.f;
    yb[q] = RV(q) ? 0.f : 1.f;
  }
#pragma unroll
  for (int i = 0; i < MAXH; ++i) {
    if (i < nh) {
      const float Fi = Fl[i];
      const float* crow = Cb + (int64_t)hidx[i] * R;
#pragma unroll
      for (int c = 0; c < CPL; ++c) kset(i, c, CV(c) ? fexp2(Fi - crow[CJ(c)] * kappa) : 0.f);
    } else {
#pragma unroll
      for (int c = 0; c < CPL; ++c) kset(i, c, 0.f);
    }
  }

  for (int32_t it = 1; it <= p.iters; ++it) {
    if (it > 1) {
      // ---- row half-step: u_i = s~_i / sum_c Kt_ic v_c ------------------------------
      uint32_t lo = 0xFFFFFFFFu, hi = 0u;  // range of the scalings' bit patterns
#pragma unroll
      for (int q = 0; q < C8; ++q) {
        float pp[8];
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          float acc = kget(8 * q + r, 0) * v[0];
#pragma unroll
          for (int c = 1; c < CPL; ++c) acc = __builtin_fmaf(kget(8 * q + r, c), v[c], acc);
          pp[r] = acc;
        }
        const float y = reduce8(pp, lane);
        const float un = sAl[8 * q + (lane >> 3)] * frcp(y + yb[q]);
        const uint32_t bits = __float_as_uint(un + yb[q]);
        lo = bits < lo ? bits : lo;
        hi = bits > hi ? bits : hi;
        uq[q] = un;
      }
      // outside [kLo, kHi], negative, infinite or NaN
      const bool fail = !(lo >= __float_as_uint(kLo) && hi <= __float_as_uint(kHi));
      if (__ballot(fail) != 0) {
        // exact log-domain update of every row, absorbed into F
#pragma unroll
        for (int i = 0; i < MAXH; ++i) {
          if (i < nh) {
            const float* crow = Cb + (int64_t)hidx[i] * R;
            float t[CPL];
            float mx = -INFINITY;
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
              t[c] = CV(c) ? (G[c] + flog2(v[c])) - crow[CJ(c)] * kappa : -INFINITY;
              mx = fmaxf(mx, t[c]);
            }
            mx = wave_max(mx);
            float sum = 0.f;
#pragma unroll
            for (int c = 0; c < CPL; ++c) sum += CV(c) ? fexp2(t[c] - mx) : 0.f;
            sum = first_lane(wave_sum(sum));
            const float fi = flog2(sAl[i]) - (mx + flog2(sum));
#pragma unroll
            for (int c = 0; c < CPL; ++c) kset(i, c, CV(c) ? fexp2((fi + G[c]) - crow[CJ(c)] * kappa) : 0.f);
            if (lane == 0) Fl[i] = fi;
          }
        }
#pragma unroll
        for (int q = 0; q < C8; ++q) uq[q] = RV(q) ? 1.f : 0.f;
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
      }
    }
    // ---- column half-step: v_c = d_c / sum_i u_i Kt_ic -------------------------------
    // the row scalings reach every lane through LDS (one store per row, two
    // broadcast 16-byte loads per 8 rows; a wave's LDS accesses run in order)
#pragma unroll
    for (int q = 0; q < C8; ++q)
      if ((lane & 7) == 0) ul[8 * q + (lane >> 3)] = uq[q];
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    float x[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) x[c] = xb[c];
#pragma unroll
    for (int q = 0; q < C8; ++q) {
      const float4 ua = *reinterpret_cast<const float4*>(ul + 8 * q);
      const float4 ub = *reinterpret_cast<const float4*>(ul + 8 * q + 4);
      const float us[8] = {ua.x, ua.y, ua.z, ua.w, ub.x, ub.y, ub.z, ub.w};
#pragma unroll
      for (int r = 0; r < 8; ++r)
#pragma unroll
        for (int c = 0; c < CPL; ++c) x[c] = __builtin_fmaf(us[r], kget(8 * q + r, c), x[c]);
    }
    uint32_t clo = 0xFFFFFFFFu, chi = 0u;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const float vn = sB[c] * frcp(x[c]);
      const uint32_t bits = __float_as_uint(vn + xb[c]);
      clo = bits < clo ? bits : clo;
      chi = bits > chi ? bits : chi;
      v[c] = vn;
    }
    const bool failc = !(clo >= __float_as_uint(kLo) && chi <= __float_as_uint(kHi));
    if (__ballot(failc) != 0) {
      // exact log-domain update of every column, absorbed into G (online LSE)
      float mx[CPL], sum[CPL];
#pragma unroll
      for (int c = 0; c < CPL; ++c) { mx[c] = -INFINITY; sum[c] = 0.f; }
#pragma unroll
      for (int i = 0; i < MAXH; ++i) {
        if (i < nh) {
          const float fi = Fl[i] + flog2(bcast(uq[i / 8], 8 * (i % 8)));
          const float* crow = Cb + (int64_t)hidx[i] * R;
#pragma unroll
          for (int c = 0; c < CPL; ++c) {
            if (CV(c)) {
              const float t = fi - crow[CJ(c)] * kappa;
              const float m2 = fmaxf(mx[c], t);
              sum[c] = sum[c] * fexp2(mx[c] - m2) + fexp2(t - m2);
              mx[c] = m2;
            }
          }
        }
      }
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        G[c] = CV(c) ? flog2(sB[c]) - (mx[c] + flog2(sum[c])) : 0.f;
        v[c] = CV(c) ? 1.f : 0.f;
      }
#pragma unroll
      for (int i = 0; i < MAXH; ++i) {
        if (i < nh) {
          const float Fi = Fl[i];
          const float* crow = Cb + (int64_t)hidx[i] * R;
#pragma unroll
          for (int c = 0; c < CPL; ++c) kset(i, c, CV(c) ? fexp2((Fi + G[c]) - crow[CJ(c)] * kappa) : 0.f);
        }
      }
    }
  }

  // ---- plan, column cap, outputs -------------------------------------------------
  const bool colcap = !(p.flags & TAOT_SK_NO_COLCAP);
  float fac[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) fac[c] = 1.f;
  if (colcap) {
    float cs[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) cs[c] = 0.f;
#pragma unroll
    for (int i = 0; i < MAXH; ++i) {
      const float ui = bcast(uq[i / 8], 8 * (i % 8));
#pragma unroll
      for (int c = 0; c < CPL; ++c) cs[c] += ui * kget(i, c) * v[c];
    }
#pragma unroll
    for (int c = 0; c < CPL; ++c) fac[c] = CV(c) ? fminf(1.f, sB[c] / (cs[c] + 1e-12f)) : 1.f;
  }
#pragma unroll
  for (int q = 0; q < C8; ++q)
    if ((lane & 7) == 0 && RV(q)) ul[8 * q + (lane >> 3)] = uq[q];
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  if (p.T) {
    float* Tb = p.T + pb * R * R;
    for (int32_t i = 0; i < R; ++i) {
      const bool hot = hpos[i] >= 0;
      for (int32_t j = lane; j < R; j += kWave)
        if (!hot || cpos[j] < 0) Tb[(int64_t)i * R + j] = 0.f;
    }
#pragma unroll
    for (int i = 0; i < MAXH; ++i) {
      if (i < nh) {
        const float ui = bcast(uq[i / 8], 8 * (i % 8));
        float* trow = Tb + (int64_t)hidx[i] * R;
#pragma unroll
        for (int c = 0; c < CPL; ++c)
          if (CV(c)) trow[CJ(c)] = ui * kget(i, c) * (v[c] * fac[c]);
      }
    }
  }
  const float to_nat = p.eps * kLn2;
  for (int32_t i = lane; i < R; i += kWave) {
    const int32_t ih = hpos[i];
    if (p.f) p.f[pb * R + i] = ih >= 0 ? (Fl[ih] + flog2(ul[ih])) * to_nat : -INFINITY;
    if (p.g && cpos[i] < 0) p.g[pb * R + i] = -INFINITY;
  }
  if (p.g) {
#pragma unroll
    for (int c = 0; c < CPL; ++c)
      if (CV(c)) p.g[pb * R + CJ(c)] = (G[c] + flog2(v[c])) * to_nat;
  }
  if (lane == 0 && p.status) p.status[pb] = 0u;
#undef RV
#undef CJ
#undef CV
}

// Two waves per problem where the row block does not fit one wave's
// registers (|H| > 48 at CPL = 4): wave w holds rows 32w .. 32w+31 and all of
// the lane's columns.  Row sums stay within a wave.  Each column half-step
// adds the two waves' partial sums in a fixed order after an exchange through
// LDS (one barrier per iteration, buffers alternating by parity), so both
// waves derive the same v and take the same branches.
template <int CPL, int C8W>
__device__ __forceinline__ void wave2_solve(const SkParams& p, int64_t pb, int32_t nh, int32_t nc,
                                            const int32_t* cpos, const int32_t* hpos, const int32_t* cidx,
                                            const int32_t* hidx, const float* sAl, float* Fl, float* ul,
                                            float* xbuf, float kappa) {
  constexpr int MW = 8 * C8W;  // rows per wave
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  const int rb = MW * wv;      // first row of this wave
  const int32_t R = p.R;
  const float* bd = p.b + pb * R;
  const float* Cb = p.C + pb * p.C_stride;
  float K[MW][CPL];
#define CV(c) (lane + kWave * (c) < nc)
#define CJ(c) (CV(c) ? cidx[lane + kWave * (c)] : 0)
#define RV(q) (rb + 8 * (q) + (lane >> 3) < nh)
  float sB[CPL], G[CPL], v[CPL], xb[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    sB[c] = CV(c) ? bd[CJ(c)] : 0.f;
    G[c] = 0.f;
    v[c] = CV(c) ? 1.f : 0.f;
    xb[c] = CV(c) ? 0.f : 1.f;
  }
  float uq[C8W], yb[C8W];
#pragma unroll
  for (int q = 0; q < C8W; ++q) {
    uq[q] = RV(q) ? 1.f : 0.f;
    yb[q] = RV(q) ? 0.f : 1.f;
  }
#pragma unroll
  for (int i = 0; i < MW; ++i) {
    const int gi = rb + i;
    if (gi < nh) {
      const float Fi = Fl[gi];
      const float* crow = Cb + (int64_t)hidx[gi] * R;
#pragma unroll
      for (int c = 0; c < CPL; ++c) K[i][c] = CV(c) ? fexp2(Fi - crow[CJ(c)] * kappa) : 0.f;
    } else {
#pragma unroll
      for (int c = 0; c < CPL; ++c) K[i][c] = 0.f;
    }
  }

  for (int32_t it = 1; it <= p.iters; ++it) {
    if (it > 1) {
      // ---- row half-step on this wave's rows ----------------------------------------
      uint32_t lo = 0xFFFFFFFFu, hi = 0u;
#pragma unroll
      for (int q = 0; q < C8W; ++q) {
        float pp[8];
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          float acc = K[8 * q + r][0] * v[0];
#pragma unroll
          for (int c = 1; c < CPL; ++c) acc = __builtin_fmaf(K[8 * q + r][c], v[c], acc);
          pp[r] = acc;
        }
        const float y = reduce8(pp, lane);
        const float un = sAl[rb + 8 * q + (lane >> 3)] * frcp(y + yb[q]);
        const uint32_t bits = __float_as_uint(un + yb[q]);
        lo = bits < lo ? bits : lo;
        hi = bits > hi ? bits : hi;
        uq[q] = un;
      }
      const bool fail = !(lo >= __float_as_uint(kLo) && hi <= __float_as_uint(kHi));
      if (__ballot(fail) != 0) {
        // exact log-domain update of this wave's rows, absorbed into F
#pragma unroll
        for (int i = 0; i < MW; ++i) {
          const int gi = rb + i;
          if (gi < nh) {
            const float* crow = Cb + (int64_t)hidx[gi] * R;
            float t[CPL];
            float mx = -INFINITY;
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
              t[c] = CV(c) ? (G[c] + flog2(v[c])) - crow[CJ(c)] * kappa : -INFINITY;
              mx = fmaxf(mx, t[c]);
            }
            mx = wave_max(mx);
            float sum = 0.f;
#pragma unroll
            for (int c = 0; c < CPL; ++c) sum += CV(c) ? fexp2(t[c] - mx) : 0.f;
            sum = first_lane(wave_sum(sum));
            const float fi = flog2(sAl[gi]) - (mx + flog2(sum));
#pragma unroll
            for (int c = 0; c < CPL; ++c) K[i][c] = CV(c) ? fexp2((fi + G[c]) - crow[CJ(c)] * kappa) : 0.f;
            if (lane == 0) Fl[gi] = fi;
          }
        }
#pragma unroll
        for (int q = 0; q < C8W; ++q) uq[q] = RV(q) ? 1.f : 0.f;
      }
    }
    // ---- column half-step: partial sums of both waves, added in wave order ------------
    // row scalings to every lane through this wave's part of ul (as in wave_solve)
#pragma unroll
    for (int q = 0; q < C8W; ++q)
      if ((lane & 7) == 0) ul[rb + 8 * q + (lane >> 3)] = uq[q];
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    float x[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) x[c] = wv == 0 ? xb[c] : 0.f;
#pragma unroll
    for (int q = 0; q < C8W; ++q) {
      const float4 ua = *reinterpret_cast<const float4*>(ul + rb + 8 * q);
      const float4 ub = *reinterpret_cast<const float4*>(ul + rb + 8 * q + 4);
      const float us[8] = {ua.x, ua.y, ua.z, ua.w, ub.x, ub.y, ub.z, ub.w};
#pragma unroll
      for (int r = 0; r < 8; ++r)
#pragma unroll
        for (int c = 0; c < CPL; ++c) x[c] = __builtin_fmaf(us[r], K[8 * q + r][c], x[c]);
    }
    float* xs = xbuf + (size_t)((it & 1) * 2 + wv) * CPL * kWave;
#pragma unroll
    for (int c = 0; c < CPL; ++c) xs[c * kWave + lane] = x[c];
    __syncthreads();
    const float* x0 = xbuf + (size_t)((it & 1) * 2) * CPL * kWave;
    const float* x1 = x0 + CPL * kWave;
#pragma unroll
    for (int c = 0; c < CPL; ++c) x[c] = x0[c * kWave + lane] + x1[c * kWave + lane];
    uint32_t clo = 0xFFFFFFFFu, chi = 0u;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const float vn = sB[c] * frcp(x[c]);
      const uint32_t bits = __float_as_uint(vn + xb[c]);
      clo = bits < clo ? bits : clo;
      chi = bits > chi ? bits : chi;
      v[c] = vn;
    }
    const bool failc = !(clo >= __float_as_uint(kLo) && chi <= __float_as_uint(kHi));
    if (__ballot(failc) != 0) {  // the same decision on both waves
      // exact log-domain update of every column, absorbed into G (online LSE
      // over all rows: each wave publishes its row scalings first)
#pragma unroll
      for (int q = 0; q < C8W; ++q)
        if ((lane & 7) == 0 && RV(q)) ul[rb + 8 * q + (lane >> 3)] = uq[q];
      __syncthreads();
      float mx[CPL], sum[CPL];
#pragma unroll
      for (int c = 0; c < CPL; ++c) { mx[c] = -INFINITY; sum[c] = 0.f; }
      for (int32_t i = 0; i < nh; ++i) {
        const float fi = Fl[i] + flog2(ul[i]);
        const float* crow = Cb + (int64_t)hidx[i] * R;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          if (CV(c)) {
            const float t = fi - crow[CJ(c)] * kappa;
            const float m2 = fmaxf(mx[c], t);
            sum[c] = sum[c] * fexp2(mx[c] - m2) + fexp2(t - m2);
            mx[c] = m2;
          }
        }
      }
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        G[c] = CV(c) ? flog2(sB[c]) - (mx[c] + flog2(sum[c])) : 0.f;
        v[c] = CV(c) ? 1.f : 0.f;
      }
#pragma unroll
      for (int i = 0; i < MW; ++i) {
        const int gi = rb + i;
        if (gi < nh) {
          const float Fi = Fl[gi];
          const float* crow = Cb + (int64_t)hidx[gi] * R;
#pragma unroll
          for (int c = 0; c < CPL; ++c) K[i][c] = CV(c) ? fexp2((Fi + G[c]) - crow[CJ(c)] * kappa) : 0.f;
        }
      }
      __syncthreads();  // both waves have read ul
    }
  }

  // ---- plan, column cap, outputs -------------------------------------------------
  const bool colcap = !(p.flags & TAOT_SK_NO_COLCAP);
  float fac[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) fac[c] = 1.f;
  if (colcap) {
    float cs[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) cs[c] = 0.f;
#pragma unroll
    for (int i = 0; i < MW; ++i) {
      const float ui = bcast(uq[i / 8], 8 * (i % 8));
#pragma unroll
      for (int c = 0; c < CPL; ++c) cs[c] += ui * K[i][c] * v[c];
    }
    // the iteration loop's last exchange used parity iters & 1
    float* xs = xbuf + (size_t)(((p.iters + 1) & 1) * 2 + wv) * CPL * kWave;
#pragma unroll
    for (int c = 0; c < CPL; ++c) xs[c * kWave + lane] = cs[c];
    __syncthreads();
    const float* c0 = xbuf + (size_t)(((p.iters + 1) & 1) * 2) * CPL * kWave;
    const float* c1 = c0 + CPL * kWave;
#pragma unroll
    for (int c = 0; c < CPL; ++c)
      fac[c] = CV(c) ? fminf(1.f, sB[c] / ((c0[c * kWave + lane] + c1[c * kWave + lane]) + 1e-12f)) : 1.f;
  }
#pragma unroll
  for (int q = 0; q < C8W; ++q)
    if ((lane & 7) == 0 && RV(q)) ul[rb + 8 * q + (lane >> 3)] = uq[q];
  __syncthreads();
  if (p.T) {
    float* Tb = p.T + pb * R * R;
    for (int32_t i = wv; i < R; i += 2) {
      const bool hot = hpos[i] >= 0;
      for (int32_t j = lane; j < R; j += kWave)
        if (!hot || cpos[j] < 0) Tb[(int64_t)i * R + j] = 0.f;
    }
#pragma unroll
    for (int i = 0; i < MW; ++i) {
      const int gi = rb + i;
      if (gi < nh) {
        const float ui = bcast(uq[i / 8], 8 * (i % 8));
        float* trow = Tb + (int64_t)hidx[gi] * R;
#pragma unroll
        for (int c = 0; c < CPL; ++c)
          if (CV(c)) trow[CJ(c)] = ui * K[i][c] * (v[c] * fac[c]);
      }
    }
  }
  if (wv == 0) {
    const float to_nat = p.eps * kLn2;
    for (int32_t i = lane; i < R; i += kWave) {
      const int32_t ih = hpos[i];
      if (p.f) p.f[pb * R + i] = ih >= 0 ? (Fl[ih] + flog2(ul[ih])) * to_nat : -INFINITY;
      if (p.g && cpos[i] < 0) p.g[pb * R + i] = -INFINITY;
    }
    if (p.g) {
#pragma unroll
      for (int c = 0; c < CPL; ++c)
        if (CV(c)) p.g[pb * R + CJ(c)] = (G[c] + flog2(v[c])) * to_nat;
    }
    if (lane == 0 && p.status) p.status[pb] = 0u;
  }
#undef RV
#undef CJ
#undef CV
}

// LDS of the wave kernels: sA, F, u [64] floats, for the two-wave solver the
// column exchange [2 parities][2 waves][4][64] floats, then cpos, hpos [R] +
// cidx [256] + hidx [64] ints.
__host__ __device__ constexpr size_t wave_lds_bytes(int32_t R, bool two) {
  return (size_t)(2 * R + 256 + 64) * 4 + 3 * 64 * 4 + (two ? (size_t)2 * 2 * 4 * kWave * 4 : 0);
}
__host__ __device__ constexpr bool two_wave_class(int cls) {
  return cls == wave_class(4, 7) || cls == wave_class(4, 8);
}

// Problem pb on one wave (TWO = false: the row block fits one wave's
// registers) or on a two-wave workgroup (TWO = true: the rest of the register
// classes); returns at once for the other kind.  Uniform over the workgroup.
template <bool TWO>
__device__ __forceinline__ void wave_problem(const SkParams& p, int64_t pb, int32_t* wl) {
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t R = p.R;
  // float arrays first: ul is read 16 bytes at a time
  float* sAl = reinterpret_cast<float*>(wl);  // [64] scaled supply
  float* Fl = sAl + 64;            // [64] absorbed row potentials (log2 units)
  float* ul = Fl + 64;             // [64] row scalings (broadcast, final, exchanges)
  float* xbuf = ul + 64;           // [2][2][4][64] column partial sums (TWO only)
  int32_t* cpos = reinterpret_cast<int32_t*>(TWO ? xbuf + 2 * 2 * 4 * kWave : xbuf);  // [R] compact column, -1 if not cold
  int32_t* hpos = cpos + R;        // [R] compact row of rank i, -1 if not hot
  int32_t* cidx = hpos + R;        // [256]
  int32_t* hidx = cidx + 256;      // [64]
  const float* a = p.a + pb * R;
  const float* bd = p.b + pb * R;
  const float* Cb = p.C + pb * p.C_stride;

  // ---- supports, validation, mass -------------------------------------------
  double sa = 0.0, sd = 0.0;
  bool bad = false;
  int32_t nh = 0, nc = 0;
  for (int32_t base = 0; base < R; base += kWave) {
    const int32_t i = base + lane;
    const bool in = i < R;
    const float ai = in ? a[i] : 0.f, bi = in ? bd[i] : 0.f;
    bad |= !(ai >= 0.f && ai <= 3.402823466e38f) || !(bi >= 0.f && bi <= 3.402823466e38f);
    sa += (double)ai;
    sd += (double)bi;
    const uint64_t hm = __ballot(in && ai > 0.f), cm = __ballot(in && bi > 0.f);
    const uint64_t below = (1ull << lane) - 1ull;
    const int32_t ph = nh + __popcll(hm & below), pc = nc + __popcll(cm & below);
    if (in) {
      hpos[i] = ai > 0.f ? ph : -1;
      cpos[i] = bi > 0.f ? pc : -1;
    }
    if (in && ai > 0.f && ph < 64) hidx[ph] = i;
    if (in && bi > 0.f && pc < 256) cidx[pc] = i;
    nh += __popcll(hm);
    nc += __popcll(cm);
  }
  const int cls = __ballot(bad) != 0 ? 0 : classify(nh, nc, p.flags);
  if (cls == 0 || two_wave_class(cls) != TWO) return;  // uniform: another kernel owns this problem
  sa = wave_sum_d(sa);
  sd = wave_sum_d(sd);
  double gamma = __shfl(sd, 0, kWave) / fmax(__shfl(sa, 0, kWave), kEps0);
  gamma = gamma < 1.0 ? gamma : 1.0;
  sAl[lane] = lane < nh ? (float)(gamma * (double)a[hidx[lane]]) : 0.f;  // zero padding to 64 rows
  __syncthreads();
  const float kappa = kLog2e / p.eps;

  // ---- first row update over all R columns (v = 1): F_i = log2 s~_i - LSE2_j(-C'_ij)
  bool badc = false;
  for (int32_t i = 0; i < nh; ++i) {
    const float* crow = Cb + (int64_t)hidx[i] * R;
    float mx = -INFINITY;
    for (int32_t j = lane; j < R; j += kWave) {
      const float c = crow[j];
      badc |= !(c == c) || c == INFINITY || c == -INFINITY;
      mx = fmaxf(mx, -c * kappa);
    }
    mx = wave_max(mx);
    float sum = 0.f;
    for (int32_t j = lane; j < R; j += kWave) sum += fexp2(-crow[j] * kappa - mx);
    sum = first_lane(wave_sum(sum));
    if (lane == 0) Fl[i] = flog2(sAl[i]) - (mx + flog2(sum));
  }
  if (__ballot(badc) != 0) {
    if (p.T)
      for (int64_t q = lane; q < (int64_t)R * R; q += kWave) p.T[pb * R * R + q] = 0.f;
    for (int32_t i = lane; i < R; i += kWave) {
      if (p.f) p.f[pb * R + i] = -INFINITY;
      if (p.g) p.g[pb * R + i] = -INFINITY;
    }
    if (lane == 0 && p.status) p.status[pb] = TAOT_ST_BAD_INPUT;
    return;
  }
  __syncthreads();
  if constexpr (TWO) {
    wave2_solve<4, 4>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, xbuf, kappa);
    return;
  } else {
  switch (cls) {
#define TAOT_WAVE_CASE(CPL_, C8_)                                                                      \
  case wave_class(CPL_, C8_):                                                                          \
    wave_solve<CPL_, C8_>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, kappa);                   \
    break;
#define TAOT_WAVE_CPL(CPL_)                                                                            \
  TAOT_WAVE_CASE(CPL_, 1) TAOT_WAVE_CASE(CPL_, 2) TAOT_WAVE_CASE(CPL_, 3) TAOT_WAVE_CASE(CPL_, 4)      \
  TAOT_WAVE_CASE(CPL_, 5) TAOT_WAVE_CASE(CPL_, 6) TAOT_WAVE_CASE(CPL_, 7) TAOT_WAVE_CASE(CPL_, 8)
    TAOT_WAVE_CPL(1) TAOT_WAVE_CPL(2)
    TAOT_WAVE_CASE(4, 1) TAOT_WAVE_CASE(4, 2) TAOT_WAVE_CASE(4, 3) TAOT_WAVE_CASE(4, 4)
    TAOT_WAVE_CASE(4, 5) TAOT_WAVE_CASE(4, 6)
#undef TAOT_WAVE_CPL
#undef TAOT_WAVE_CASE
    default: break;
  }
  }
}

__global__ void __launch_bounds__(kWave, 2)
sinkhorn_wave_kernel(SkParams p, const int32_t* __restrict__ ord, const int32_t* __restrict__ count) {
  extern __shared__ __attribute__((aligned(16))) int32_t wl[];
  if ((int32_t)blockIdx.x >= *count) return;
  wave_problem<false>(p, ord[blockIdx.x], wl);
}

// The listed two-wave problems, a small grid walking the list.
__global__ void __launch_bounds__(2 * kWave, 2)
sinkhorn_wave2_kernel(SkParams p, const int32_t* __restrict__ list, const int32_t* __restrict__ count) {
  extern __shared__ __attribute__((aligned(16))) int32_t wl[];
  const int32_t n = *count;
  for (int32_t k = blockIdx.x; k < n; k += gridDim.x) {
    wave_problem<true>(p, list[k], wl);
    __syncthreads();  // LDS is reused by the next problem
  }
}

// Register class of every problem (0: not a register problem), with the same
// support scan and tests as wave_problem.
__global__ void __launch_bounds__(kWave) wave_class_kernel(SkParams p, int32_t* __restrict__ cls) {
  const int lane = threadIdx.x;
  const int64_t pb = blockIdx.x;
  const int32_t R = p.R;
  const float* a = p.a + pb * R;
  const float* bd = p.b + pb * R;
  bool bad = false;
  int32_t nh = 0, nc = 0;
  for (int32_t base = 0; base < R; base += kWave) {
    const int32_t i = base + lane;
    const bool in = i < R;
    const float ai = in ? a[i] : 0.f, bi = in ? bd[i] : 0.f;
    bad |= !(ai >= 0.f && ai <= 3.402823466e38f) || !(bi >= 0.f && bi <= 3.402823466e38f);
    nh += __popcll(__ballot(in && ai > 0.f));
    nc += __popcll(__ballot(in && bi > 0.f));
  }
  const int c = __ballot(bad) != 0 ? 0 : classify(nh, nc, p.flags);
  if (lane == 0) cls[pb] = c;
}

// Per-iteration work of a register class: rows (8 C8) x columns per lane.
__device__ __forceinline__ int32_t class_work(int32_t cls) {
  const int32_t c8 = (cls - 1) % 8 + 1, ci = (cls - 1) / 8;
  return c8 * (ci == 0 ? 1 : ci == 1 ? 2 : 4);
}

// Launch orders (one block): the two-wave problems ascending, and the
// one-wave problems by descending work (ascending index within equal work),
// so that workgroups dealt out in order mix heavy and light problems on every
// compute unit.
__global__ void __launch_bounds__(kSkThreads) wave_order_kernel(const int32_t* __restrict__ cls, int32_t B,
                                                                int32_t* __restrict__ list2,
                                                                int32_t* __restrict__ count2,
                                                                int32_t* __restrict__ ord1,
                                                                int32_t* __restrict__ count1) {
  __shared__ int32_t wave_cnt[kSkWaves];
  __shared__ unsigned long long present;  // bit w: some one-wave problem has work w
  if (threadIdx.x == 0) present = 0ull;
  __syncthreads();
  for (int32_t b = threadIdx.x; b < B; b += kSkThreads) {
    const int32_t c = cls[b];
    if (c != 0 && !two_wave_class(c)) atomicOr(&present, 1ull << class_work(c));
  }
  __syncthreads();
  const unsigned long long works = present;
  int32_t n = 0;
  for (int32_t base = 0; base < B; base += kSkThreads) {
    const int32_t b = base + (int32_t)threadIdx.x;
    const bool f = b < B && two_wave_class(cls[b]);
    int32_t tot;
    const int32_t pos = chunk_compact(f, wave_cnt, tot);
    if (f) list2[n + pos] = b;
    n += tot;
  }
  if (threadIdx.x == 0) *count2 = n;
  n = 0;
  for (int32_t wk = 63; wk > 0; --wk) {
    if (!((works >> wk) & 1ull)) continue;
    for (int32_t base = 0; base < B; base += kSkThreads) {
      const int32_t b = base + (int32_t)threadIdx.x;
      const int32_t c = b < B ? cls[b] : 0;
      const bool f = c != 0 && !two_wave_class(c) && class_work(c) == wk;
      int32_t tot;
      const int32_t pos = chunk_compact(f, wave_cnt, tot);
      if (f) ord1[n + pos] = b;
      n += tot;
    }
  }
  if (threadIdx.x == 0) *count1 = n;
}

// A stream beside the caller's, so that the one- and two-wave kernels run
// concurrently: created once per device and kept for the life of the
// process, at the default priority.
struct SideStream {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};
constexpr int kMaxDevices = 64;
constexpr int kTwoWaveGrid = 64;  // workgroups of the two-wave kernel
std::mutex g_side_mutex;
SideStream g_side[kMaxDevices];

// The register path: classes and the two-wave list on the caller's stream;
// then the two-wave kernel (a small grid, launched first so that its
// workgroups find room) on the caller's stream, beside the one-wave kernel on
// the side stream; the caller's stream waits for both.
taot_status launch_wave(const SkParams& p, int32_t* cls, int32_t* list, int32_t* count, int32_t* ord,
                        int32_t* count1, hipStream_t stream) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return TAOT_ERR_LAUNCH;
  hipLaunchKernelGGL(wave_class_kernel, dim3((unsigned)p.B), dim3(kWave), 0, stream, p, cls);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  hipLaunchKernelGGL(wave_order_kernel, dim3(1), dim3(kSkThreads), 0, stream, cls, p.B, list, count, ord, count1);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  std::lock_guard<std::mutex> lock(g_side_mutex);
  SideStream& sd = g_side[dev];
  if (sd.s == nullptr) {
    if (hipStreamCreateWithFlags(&sd.s, hipStreamNonBlocking) != hipSuccess ||
        hipEventCreateWithFlags(&sd.fork, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&sd.join, hipEventDisableTiming) != hipSuccess)
      return TAOT_ERR_LAUNCH;
  }
  if (hipEventRecord(sd.fork, stream) != hipSuccess) return TAOT_ERR_LAUNCH;
  const unsigned grid2 = (unsigned)(p.B < kTwoWaveGrid ? p.B : kTwoWaveGrid);
  hipLaunchKernelGGL(sinkhorn_wave2_kernel, dim3(grid2), dim3(2 * kWave), wave_lds_bytes(p.R, true), stream, p,
                     list, count);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  if (hipStreamWaitEvent(sd.s, sd.fork, 0) != hipSuccess) return TAOT_ERR_LAUNCH;
  hipLaunchKernelGGL(sinkhorn_wave_kernel, dim3((unsigned)p.B), dim3(kWave), wave_lds_bytes(p.R, false), sd.s, p,
                     ord, count1);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  if (hipEventRecord(sd.join, sd.s) != hipSuccess) return TAOT_ERR_LAUNCH;
  return hipStreamWaitEvent(stream, sd.join, 0) == hipSuccess ? TAOT_OK : TAOT_ERR_LAUNCH;
}

// Largest nh * nc over disjoint supports of R ranks (nh + nc <= R).
int64_t max_block(int32_t R) { return (int64_t)(R / 2) * (R - R / 2); }

struct SkWs {
  int32_t* flag;
  int32_t* cls;    // [B] register class
  int32_t* list;   // [B] two-wave problems
  int32_t* count;  // [1]
  int32_t* ord;    // [B] one-wave problems by descending work
  int32_t* count1; // [1]
  float* kt;
  int64_t kt_stride;
  size_t bytes;
};

SkWs carve(void* ws, int32_t B, int32_t R) {
  Carver c{static_cast<char*>(ws)};
  SkWs w;
  w.flag = c.take<int32_t>((size_t)B);
  w.cls = c.take<int32_t>((size_t)B);
  w.list = c.take<int32_t>((size_t)B);
  w.count = c.take<int32_t>(1);
  w.ord = c.take<int32_t>((size_t)B);
  w.count1 = c.take<int32_t>(1);
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
  if (!(flags & (TAOT_SK_FORCE_STREAM | TAOT_SK_NO_REGISTER))) {
    const taot_status st = launch_wave(p, w.cls, w.list, w.count, w.ord, w.count1, stream);
    if (st != TAOT_OK) return st;
  }
  if (lds_path) {
    p.lds_kt_cap = (int32_t)max_block(R);
    const size_t lds = vec_bytes + (size_t)p.lds_kt_cap * sizeof(float);
    if (lds > 65536 && hipFuncSetAttribute((const void*)sinkhorn_kernel<false, kSkThreads>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)lds) != hipSuccess)
      return TAOT_ERR_LAUNCH;
    hipLaunchKernelGGL((sinkhorn_kernel<false, kSkThreads>), dim3((unsigned)B), dim3(kSkThreads), lds, stream, p);
    if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  } else {
    p.all_streamed = 1;
  }
  if (vec_bytes > 65536 && hipFuncSetAttribute((const void*)sinkhorn_kernel<true, kSkStreamThreads>,
                                               hipFuncAttributeMaxDynamicSharedMemorySize,
                                               (int)vec_bytes) != hipSuccess)
    return TAOT_ERR_LAUNCH;
  hipLaunchKernelGGL((sinkhorn_kernel<true, kSkStreamThreads>), dim3((unsigned)B), dim3(kSkStreamThreads), vec_bytes,
                     stream, p);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  return TAOT_OK;
}

}  // namespace taot
