// Step 3 of the planner: batched Phase-1 Sinkhorn-Knopp (Sec. A.2).
//
// The paper's iteration is the linear-domain pair u = s~ / (M v),
// v = d / (M^T u) with M = exp(-C / eps), T = diag(u) M diag(v).  In fp32 the
// kernel M underflows for the costs used here (exp(-8 / 0.08)), so the
// iterate is carried in the stabilised form of Schmitzer (2019, "Stabilized
// sparse scaling algorithms for entropy regularized transport problems"):
//     T = diag(u) Kt diag(v),  Kt_ij = exp2(F_i + G_j - C'_ij),  C' = C log2(e) / eps,
// where F, G are absorbed potentials (log2 units) and u, v are scalings kept
// in [2^-60, 2^60].  One half-step is one GEMV-like sweep with one FMA per
// entry; when a scaling leaves its range (or its sum under/overflows) that
// row or column is recomputed exactly in the log domain (max-shifted
// log-sum-exp over the current potentials), absorbed into F or G and its Kt
// entries rebuilt.  In exact arithmetic this is the same iterate as the
// paper's update; the fp32 result agrees with the fp64 definition to
// rounding.  The range is wide to keep the (costly) log-domain updates rare,
// and narrow enough that a Kt entry lost to underflow (below 2^-149) carries
// less than 2^-29 of plan mass (u v < 2^120).  A sum that overflows or
// underflows gives an out-of-range scaling and so takes the exact update.
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
#include <algorithm>

#include "common.h"

namespace taot {
namespace {

constexpr int kSkThreads = 256;
constexpr int kSkWaves = kSkThreads / kWave;
constexpr int kSkStreamThreads = 1024;  // threads per problem of the streamed kernel
constexpr float kLo = 0x1p-60f;
constexpr float kHi = 0x1p60f;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kLdsMaxR = 256;            // beyond this every problem is streamed
constexpr int kVecArrays = 11;           // per-problem vectors of length R in LDS

__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float flog2(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float frcp(float x) { return __builtin_amdgcn_rcpf(x); }

// Register classes: CPL columns per lane (|C| <= 64*CPL) and 8*C8 rows
// (|H| <= 8*C8).  Class 0 is every other problem (degenerate, larger, or the
// register path switched off).
__host__ __device__ constexpr int cpl_index(int cpl) { return cpl == 1 ? 0 : cpl == 2 ? 1 : 2; }
__host__ __device__ constexpr int wave_class(int cpl, int c8) { return 1 + cpl_index(cpl) * 8 + (c8 - 1); }
__device__ __forceinline__ int classify(int32_t nh, int32_t nc, uint32_t flags) {
  if (nh <= 0 || nc <= 0 || nh > 64 || nc > 256) return 0;
  if (flags & (TAOT_SK_FORCE_STREAM | TAOT_SK_NO_REGISTER)) return 0;
  const int cpl = nc <= 64 ? 1 : nc <= 128 ? 2 : 4;
  return wave_class(cpl, (nh + 7) / 8);
}

// Wide register classes (see the wide register path below): up to 96 hot
// and 1024 cold ranks, for problems no register class takes.
constexpr int kWideWaves = 12;
constexpr int kWideRows = 8 * kWideWaves;  // hot ranks
constexpr int kWideMaxCpl = 16;            // LDS slots per lane
constexpr int kWideCols = 64 * 15;         // cold ranks (15 columns per lane)
constexpr int kWideThreads = kWideWaves * kWave;
constexpr int kWideClassBase = 32;         // class codes 32 + CPL

// Columns per lane: 4, an even count up to 14, or 15.
__host__ __device__ constexpr int wide_cpl(int32_t nc) {
  return nc <= 256 ? 4 : nc > 896 ? 15 : (int)((nc + 127) / 128) * 2;
}
__device__ __forceinline__ int wide_class(int32_t nh, int32_t nc, uint32_t flags) {
  if (nh <= 0 || nc <= 0 || nh > kWideRows || nc > kWideCols) return 0;
  if (flags & (TAOT_SK_FORCE_STREAM | TAOT_SK_NO_REGISTER)) return 0;
  if (classify(nh, nc, flags) != 0) return 0;  // a register class takes it
  return kWideClassBase + wide_cpl(nc);
}
__host__ __device__ constexpr bool is_reg_class(int32_t c) { return c >= 1 && c < kWideClassBase; }
__host__ __device__ constexpr bool is_wide_class(int32_t c) { return c > kWideClassBase; }

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
  const int32_t* cbad;   // [matrices][cchunks] 1 = the chunk of C holds a non-finite entry
  int32_t cchunks;       // chunks of kScanChunk entries per cost matrix
};

// Cost validation.  Every entry of a problem's C is checked (not only those
// the iterate reads): cost_scan_kernel marks each chunk of kScanChunk
// entries that holds a NaN or an infinity, once per call for a shared C and
// once per problem for per-problem costs; the class prepass and the LDS and
// streamed kernels OR the chunk marks of their problem's matrix.
constexpr int64_t kScanChunk = 65536;
constexpr int kScanThreads = 256;
__host__ __device__ constexpr int32_t scan_chunks(int32_t R) {
  return (int32_t)(((int64_t)R * R + kScanChunk - 1) / kScanChunk);
}

__global__ void __launch_bounds__(kScanThreads)
cost_scan_kernel(const float* __restrict__ C, int64_t R2, int32_t chunks, int32_t* __restrict__ cbad) {
  const int64_t mat = blockIdx.x / chunks, ch = blockIdx.x % chunks;
  const float* c = C + mat * R2;
  const int64_t lo = ch * kScanChunk, hi = lo + kScanChunk < R2 ? lo + kScanChunk : R2;
  int bad = 0;
  for (int64_t q = lo + threadIdx.x; q < hi; q += kScanThreads) {
    const float x = c[q];
    bad |= !(x - x == 0.f);  // NaN or +-inf
  }
  bad = __syncthreads_or(bad);
  if (threadIdx.x == 0) cbad[blockIdx.x] = bad ? 1 : 0;
}

// Whether problem pb's cost matrix holds a non-finite entry; the chunk marks
// are read by lane (uniform result over the wave).
__device__ __forceinline__ bool cost_bad_wave(const SkParams& p, int64_t pb) {
  const int64_t base = (p.C_stride ? pb : 0) * p.cchunks;
  bool bad = false;
  for (int32_t k = threadIdx.x & (kWave - 1); k < p.cchunks; k += kWave) bad |= p.cbad[base + k] != 0;
  return __ballot(bad) != 0;
}

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
  if (wid == 0 && cost_bad_wave(p, pb) && lane == 0) sh_bad = 1;
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
  if (!degenerate && (classify(nh, nc, p.flags) != 0 || wide_class(nh, nc, p.flags) != 0)) {  // a register path owns it
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
      for (int32_t j = lane; j < R; j += kWave) mx = fmaxf(mx, -crow[j] * kappa);
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
// Register-resident path.  A problem's |H| x |C| block of Kt lives in the
// VGPRs of NW waves of one workgroup (NW = 1, 2 or 4).  Lane l of every wave
// owns compact columns l, l+64, ... (CPL of them); wave w holds the rows of
// chunks w*C8W .. w*C8W + C8W-1 (8 rows per chunk).
//   row half-step:    p_i = sum_c Kt_ic v_c per lane, then a transposed
//                     butterfly reduce-scatter over the 64 lanes (8 rows at a
//                     time: permlane32/16 swaps, then DPP) leaves the total of
//                     row 8q + (l >> 3) in lane l; rows never leave their wave.
//   column half-step: x_c = sum_i u_i Kt_ic over the wave's rows, the row
//                     scalings broadcast through LDS; with NW > 1 the waves'
//                     partial sums meet in LDS (one barrier per iteration) and
//                     are added in wave order, so every wave derives the same
//                     v and takes the same branches.
// An out-of-range scaling triggers the exact log-domain update of the wave's
// rows (or of all columns), absorbed into the potentials, with Kt rebuilt.
//
// Launch shape.  One kernel runs every register problem of a batch.  Its
// shapes use W waves per multi-wave problem (W = 4 when the batch is small
// enough that every problem can hold four waves at once, else W = 2), and its
// workgroups run either one problem on W waves ("multi") or one problem per
// wave ("single"), never two multi-wave problems, so workgroup barriers only
// ever join the waves of one problem.  Single groups of the two-wave shapes
// span a whole compute unit (eight waves) so that the problems sharing a SIMD
// can be paired by work.
//   W = 4 (at most 128 VGPRs, four waves per SIMD): problems of one chunk are
//     single; the rest are multi with ceil(C8 / 4) chunks per wave.
//   W = 2 (at most 256 VGPRs, two waves per SIMD): a problem is single when
//     its block fits one wave's 192 Kt registers, else (4 columns per lane and
//     more than 48 hot ranks) multi with ceil(C8 / 2) chunks per wave.
// Small batches thus spread a problem over more waves (a shorter dependent
// chain per wave, more waves per SIMD), while a batch that fills the chip
// with one wave per problem avoids the per-iteration exchange.

__host__ __device__ constexpr int max_c8_single(int W, int cpl) {
  return W == 4 ? 1 : (192 / (8 * cpl) < 8 ? 192 / (8 * cpl) : 8);
}
__host__ __device__ constexpr bool is_single(int W, int cpl, int c8) { return c8 <= max_c8_single(W, cpl); }
__host__ __device__ constexpr int c8_per_wave(int W, int cpl, int c8) {
  return is_single(W, cpl, c8) ? c8 : (c8 + W - 1) / W;
}
// Shapes compiled into the W-wave kernel for NW = 1 (single) or NW = W.
__host__ __device__ constexpr bool shape_ok(int W, int nw, int cpl, int c8w) {
  return nw == 1 ? c8w >= 1 && c8w <= max_c8_single(W, cpl)
                 : nw == W && (W == 4 ? c8w >= 1 && c8w <= 2 : cpl == 4 && c8w == 4);
}
__host__ __device__ constexpr bool shapes_covered() {
  for (int W = 2; W <= 4; W += 2)
    for (int ci = 0; ci < 3; ++ci)
      for (int c8 = 1; c8 <= 8; ++c8) {
        const int cpl = 1 << ci;
        const int nw = is_single(W, cpl, c8) ? 1 : W;
        if (!shape_ok(W, nw, cpl, c8_per_wave(W, cpl, c8))) return false;
      }
  return true;
}
static_assert(shapes_covered(), "every register class must map to a compiled shape");

// Decoded register class.
__device__ __forceinline__ int class_cpl(int32_t cls) { return 1 << ((cls - 1) / 8); }
__device__ __forceinline__ int class_c8(int32_t cls) { return (cls - 1) % 8 + 1; }

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

// Max and sum over the 64 lanes, every lane getting the result (bitwise the
// same: each step combines symmetric partners): DPP steps within each
// 16-lane row, then the permlane16 and permlane32 swaps across rows.
__device__ __forceinline__ float lanes_max(float x) {
  x = fmaxf(x, dpp<0xB1>(x));   // quad_perm [1,0,3,2]
  x = fmaxf(x, dpp<0x4E>(x));   // quad_perm [2,3,0,1]
  x = fmaxf(x, dpp<0x141>(x));  // row_half_mirror
  x = fmaxf(x, dpp<0x140>(x));  // row_mirror
  float y = x;
  swap16(x, y);
  x = fmaxf(x, y);
  y = x;
  swap32(x, y);
  return fmaxf(x, y);
}
__device__ __forceinline__ float lanes_sum(float x) {
  x = x + dpp<0xB1>(x);
  x = x + dpp<0x4E>(x);
  x = x + dpp<0x141>(x);
  x = x + dpp<0x140>(x);
  float y = x;
  swap16(x, y);
  x = x + y;
  y = x;
  swap32(x, y);
  return x + y;
}

// LDS of the register kernels, per workgroup: floats sA, F, u [64], the
// waves' column potentials [NW][4][64] and column demands [NW][64][4], for
// NW > 1 the column exchange [2 parities][NW][4][64]; then ints: a flag [4],
// cpos, hpos [R], cidx [256], hidx [64].
__host__ __device__ constexpr size_t wave_lds_floats(int nw) {
  return (size_t)3 * 64 + (size_t)2 * nw * 4 * 64 + (nw > 1 ? (size_t)2 * nw * 4 * 64 : 0);
}
__host__ __device__ constexpr size_t wave_lds_bytes(int32_t R, int nw) {
  return wave_lds_floats(nw) * 4 + (size_t)(4 + 2 * R + 256 + 64) * 4;
}

// Synchronisation among the waves of one problem: the workgroup barrier when
// the problem has the whole workgroup; for a one-wave problem (possibly beside
// other one-wave problems of the workgroup) an LDS fence of the wave.
template <int NW>
__device__ __forceinline__ void psync() {
  if constexpr (NW > 1) {
    __syncthreads();
  } else {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  }
}

// Iterations and outputs of one problem on NW waves of CPL columns per lane
// and C8W chunks per wave; the caller has filled the LDS vectors and the
// first-update potentials Fl.
template <int CPL, int C8W, int NW, int WV>
__device__ __forceinline__ void wave_solve(const SkParams& p, int64_t pb, int32_t nh, int32_t nc,
                                           const int32_t* cpos, const int32_t* hpos, const int32_t* cidx,
                                           const int32_t* hidx, const float* sAl, float* Fl, float* ul,
                                           float* Gall, float* Sall, float* xbuf, float kappa) {
  constexpr int MW = 8 * C8W;  // rows per wave
  const int lane = threadIdx.x & (kWave - 1);
  constexpr int wv = WV;  // this wave (a compile-time constant, so per-wave LDS offsets are immediates)
  constexpr int rb = MW * wv;  // first row of this wave
  const int32_t R = p.R;
  const float* bd = p.b + pb * R;
  const float* Cb = p.C + pb * p.C_stride;
  // the column potentials G (log2 units) are only touched by the log-domain
  // updates: they live in this wave's LDS slice, one value per lane and column
  float* Gw = Gall + wv * 4 * kWave + lane;
  // the column demands, read once per iteration: this wave's slice, the
  // lane's CPL values contiguous
  float* Sw = Sall + (wv * kWave + lane) * 4;
#define CV(c) (lane + kWave * (c) < nc)
#define CJ(c) (CV(c) ? cidx[lane + kWave * (c)] : 0)
#define RV(q) (rb + 8 * (q) + (lane >> 3) < nh)
#define GL(c) Gw[(c) * kWave]

  float K[MW][CPL];
  float v[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    Sw[c] = CV(c) ? bd[CJ(c)] : 0.f;
    v[c] = CV(c) ? 1.f : 0.f;
    GL(c) = 0.f;
  }
  // the lane's column demands (padding columns 0)
  auto demands = [&](float (&sB)[CPL]) {
    if constexpr (CPL == 4) {
      const float4 d = *reinterpret_cast<const float4*>(Sw);
      sB[0] = d.x; sB[1] = d.y; sB[2] = d.z; sB[3] = d.w;
    } else if constexpr (CPL == 2) {
      const float2 d = *reinterpret_cast<const float2*>(Sw);
      sB[0] = d.x; sB[1] = d.y;
    } else {
      sB[0] = Sw[0];
    }
  };
  // Kt of this wave's rows from the potentials (after the exact log-domain
  // update of each row's potential when row_update is set:
  // F_i = log2 s~_i - LSE2_c(G_c + log2 v_c - C'_ic), absorbing u_i).  Each
  // row's support index is read at an opaque position, so that the row's cost
  // address is formed here and not kept in registers for the whole iteration
  // loop.
  auto build = [&](bool row_update) {
#pragma unroll
    for (int i = 0; i < MW; ++i) {
      const int gi = rb + i;
      if (gi < nh) {
        int32_t go = __builtin_amdgcn_readfirstlane(gi);
        asm volatile("" : "+s"(go));
        const float* crow = Cb + (int64_t)__builtin_amdgcn_readfirstlane(hidx[go]) * R;
        float cc[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) cc[c] = CV(c) ? crow[CJ(c)] * kappa : 0.f;
        float fi;
        if (row_update) {
          float t[CPL];
          float mx = -INFINITY;
#pragma unroll
          for (int c = 0; c < CPL; ++c) {
            t[c] = CV(c) ? (GL(c) + flog2(v[c])) - cc[c] : -INFINITY;
            mx = fmaxf(mx, t[c]);
          }
          mx = lanes_max(mx);
          float sum = 0.f;
#pragma unroll
          for (int c = 0; c < CPL; ++c) sum += CV(c) ? fexp2(t[c] - mx) : 0.f;
          sum = lanes_sum(sum);
          fi = flog2(sAl[gi]) - (mx + flog2(sum));
          if (lane == 0) Fl[gi] = fi;
        } else {
          fi = Fl[gi];
        }
#pragma unroll
        for (int c = 0; c < CPL; ++c) K[i][c] = CV(c) ? fexp2((fi + GL(c)) - cc[c]) : 0.f;
      } else {
#pragma unroll
        for (int c = 0; c < CPL; ++c) K[i][c] = 0.f;
      }
    }
  };

  // The row scalings live in LDS (ul): lane l computes that of row
  // rb + 8q + (l >> 3) of chunk q, and lanes l = 8k store them.
#define UST(q, val) \
  if ((lane & 7) == 0) ul[rb + 8 * (q) + (lane >> 3)] = (val)
#pragma unroll
  for (int q = 0; q < C8W; ++q) UST(q, RV(q) ? 1.f : 0.f);
  // the scaled supply of the lane's row of each chunk, held in registers
  float sAq[C8W];
#pragma unroll
  for (int q = 0; q < C8W; ++q) sAq[q] = sAl[rb + 8 * q + (lane >> 3)];

  // The iterations run in an inner loop that only ever reads Kt.  An
  // out-of-range scaling leaves it; the log-domain update is then taken and Kt
  // rebuilt before the iterations resume, so Kt is never live across an update.
  int32_t it = 1;
  bool skip_row = true;     // iteration 1 has no row half-step (u follows from v = 1)
  bool row_update = false;  // this wave's rows take the log-domain update first
  for (;;) {
    build(row_update);
    if (row_update) {
#pragma unroll
      for (int q = 0; q < C8W; ++q) UST(q, RV(q) ? 1.f : 0.f);
      row_update = false;
    }
    bool done = false, col_fail = false;
    for (;;) {
      if (!skip_row) {
        // ---- row half-step on this wave's rows: u_i = s~_i / sum_c Kt_ic v_c ---------
        // padding rows (all-zero Kt) divide by 1 and count as 1 in the range test
        uint32_t lo = 0xFFFFFFFFu, hi = 0u;  // range of the scalings' bit patterns
#define TAOT_ROW_SUMS(q, pp)                                                                          \
  _Pragma("unroll") for (int r = 0; r < 8; ++r) {                                                     \
    float acc = K[8 * (q) + r][0] * v[0];                                                             \
    _Pragma("unroll") for (int c = 1; c < CPL; ++c) acc = __builtin_fmaf(K[8 * (q) + r][c], v[c], acc); \
    pp[r] = acc;                                                                                      \
  }
#define TAOT_ROW_FINISH(q, y)                                                                         \
  {                                                                                                   \
    const bool rv = RV(q);                                                                            \
    const float un = sAq[q] * frcp(rv ? (y) : 1.f);                                                   \
    const uint32_t bits = __float_as_uint(rv ? un : 1.f);                                             \
    lo = bits < lo ? bits : lo;                                                                       \
    hi = bits > hi ? bits : hi;                                                                       \
    UST(q, un);                                                                                       \
  }
#pragma unroll
        for (int q = 0; q < C8W; ++q) {
          float pp[8];
          TAOT_ROW_SUMS(q, pp)
          const float y = reduce8(pp, lane);  // all lanes take part
          TAOT_ROW_FINISH(q, y)
        }
#undef TAOT_ROW_FINISH
#undef TAOT_ROW_SUMS
        // outside [kLo, kHi], negative, infinite or NaN: this wave's rows are
        // updated exactly, then the iteration continues with its column half-step
        const bool fail = !(lo >= __float_as_uint(kLo) && hi <= __float_as_uint(kHi));
        if (__ballot(fail) != 0) {
          row_update = true;
          skip_row = true;
          break;
        }
      }
      skip_row = false;
      // ---- column half-step: v_c = d_c / sum_i u_i Kt_ic -------------------------------
      // this wave's row scalings reach its lanes through LDS (two broadcast
      // 16-byte loads per 8 rows; a wave's LDS accesses run in order)
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      // two partial sums per column (even and odd rows of each chunk), so
      // that 2 CPL independent FMA chains interleave
      float x[CPL], x2[CPL];
#pragma unroll
      for (int c = 0; c < CPL; ++c) x[c] = x2[c] = 0.f;
      // the loads of chunk q + 1 are issued before chunk q's FMAs
      float4 ua = *reinterpret_cast<const float4*>(ul + rb);
      float4 ub = *reinterpret_cast<const float4*>(ul + rb + 4);
#pragma unroll
      for (int q = 0; q < C8W; ++q) {
        float4 na = ua, nb = ub;
        if (q + 1 < C8W) {
          na = *reinterpret_cast<const float4*>(ul + rb + 8 * (q + 1));
          nb = *reinterpret_cast<const float4*>(ul + rb + 8 * (q + 1) + 4);
        }
        const float us[8] = {ua.x, ua.y, ua.z, ua.w, ub.x, ub.y, ub.z, ub.w};
#pragma unroll
        for (int r = 0; r < 8; r += 2)
#pragma unroll
          for (int c = 0; c < CPL; ++c) {
            x[c] = __builtin_fmaf(us[r], K[8 * q + r][c], x[c]);
            x2[c] = __builtin_fmaf(us[r + 1], K[8 * q + r + 1][c], x2[c]);
          }
        ua = na;
        ub = nb;
      }
#pragma unroll
      for (int c = 0; c < CPL; ++c) x[c] = x[c] + x2[c];
      if constexpr (NW > 1) {
        float* xs = xbuf + (size_t)((it & 1) * NW + wv) * CPL * kWave;
#pragma unroll
        for (int c = 0; c < CPL; ++c) xs[c * kWave + lane] = x[c];
        psync<NW>();
        const float* x0 = xbuf + (size_t)(it & 1) * NW * CPL * kWave;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          float sx = x0[c * kWave + lane];
#pragma unroll
          for (int w = 1; w < NW; ++w) sx = sx + x0[(w * CPL + c) * kWave + lane];
          x[c] = sx;
        }
      }
      // padding columns (all-zero Kt) divide by 1 and count as 1 in the range test
      float sB[CPL];
      demands(sB);
      uint32_t clo = 0xFFFFFFFFu, chi = 0u;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const float vn = sB[c] * frcp(CV(c) ? x[c] : 1.f);
        const uint32_t bits = __float_as_uint(CV(c) ? vn : 1.f);
        clo = bits < clo ? bits : clo;
        chi = bits > chi ? bits : chi;
        v[c] = vn;
      }
      // the same decision on every wave
      col_fail = __ballot(!(clo >= __float_as_uint(kLo) && chi <= __float_as_uint(kHi))) != 0;
      done = it == p.iters;
      if (!done) ++it;
      if (col_fail || done) break;
    }
    if (col_fail) {
      // exact log-domain update of every column, absorbed into G (online LSE
      // over all rows, whose scalings every wave has stored in ul); Kt is
      // rebuilt at the top of the loop, or below after the last iteration
      psync<NW>();
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
      float sB[CPL];
      demands(sB);
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        GL(c) = CV(c) ? flog2(sB[c]) - (mx[c] + flog2(sum[c])) : 0.f;
        v[c] = CV(c) ? 1.f : 0.f;
      }
      psync<NW>();  // every wave has read ul and F
      if (done) {
        build(false);
        break;
      }
      continue;
    }
    if (done) break;
  }

  // ---- plan, column cap, outputs -------------------------------------------------
  psync<NW>();  // the row scalings of every wave are in ul
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
      const float ui = ul[rb + i];
#pragma unroll
      for (int c = 0; c < CPL; ++c) cs[c] += ui * K[i][c] * v[c];
    }
    if constexpr (NW > 1) {
      // the iteration loop's last exchange used parity iters & 1
      float* xs = xbuf + (size_t)(((p.iters + 1) & 1) * NW + wv) * CPL * kWave;
#pragma unroll
      for (int c = 0; c < CPL; ++c) xs[c * kWave + lane] = cs[c];
      psync<NW>();
      const float* c0 = xbuf + (size_t)((p.iters + 1) & 1) * NW * CPL * kWave;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        float s = c0[c * kWave + lane];
#pragma unroll
        for (int w = 1; w < NW; ++w) s = s + c0[(w * CPL + c) * kWave + lane];
        cs[c] = s;
      }
    }
    float sB[CPL];
    demands(sB);
#pragma unroll
    for (int c = 0; c < CPL; ++c) fac[c] = CV(c) ? fminf(1.f, sB[c] / (cs[c] + 1e-12f)) : 1.f;
  }
  if (p.T) {
    float* Tb = p.T + pb * R * R;
    for (int32_t i = wv; i < R; i += NW) {
      const bool hot = hpos[i] >= 0;
      for (int32_t j = lane; j < R; j += kWave)
        if (!hot || cpos[j] < 0) Tb[(int64_t)i * R + j] = 0.f;
    }
#pragma unroll
    for (int i = 0; i < MW; ++i) {
      const int gi = rb + i;
      if (gi < nh) {
        const float ui = ul[gi];
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
        if (CV(c)) p.g[pb * R + CJ(c)] = (GL(c) + flog2(v[c])) * to_nat;
    }
    if (lane == 0 && p.status) p.status[pb] = 0u;
  }
#undef UST
#undef GL
#undef RV
#undef CJ
#undef CV
}

// ---------------------------------------------------------------------------
// One-wave layout with the columns folded over the two half-waves.  Lane l
// sits in half h = l >> 5 at column lane cl = l & 31 and owns compact columns
// cl, cl + 32, ... (CPL of them, so the block is padded to 32-column rather
// than 64-column steps); chunk q of 8 rows keeps rows 8q .. 8q+3 in half 0
// and 8q+4 .. 8q+7 in half 1, four Kt values per column.
//   row half-step:    per-lane partial sums of the half's 4 rows, then the
//                     transposed butterfly over the 32 lanes of each half
//                     (permlane16 swap, then DPP) leaves the total of row
//                     8q + (l >> 3) in lane l, as in the full-wave layout.
//   column half-step: partial sums over the half's rows; one permlane32 swap
//                     and an add per pair of columns (c, c + P) leave the
//                     totals of column c in half 0 and of column c + P in
//                     half 1, each half derives those scalings, and a second
//                     swap hands every lane both.
// Against the full-wave layout this drops one swap level from every row
// chunk (the halves' column partials meet once per iteration instead) and
// pads the columns less.

// Sums 4 per-lane values over the 32 lanes of each half-wave; lane l ends
// with the total of value (l >> 3) & 3 of its half.  The steps pair lanes
// l ^ 16 (permlane16 swap), l <-> 15 - l (row_mirror), l <-> l ^ 7
// (row_half_mirror), l ^ 2 and l ^ 1 (quad_perm).
__device__ __forceinline__ float reduce4(float (&p)[4], int lane) {
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
// Sums 8 per-lane values over the 32 lanes of each half-wave; lane l ends
// with the total of value 4 b4 + 2 b2 + b3 of its half (bk = bit k of l).
// The steps pair lanes l ^ 16 (permlane16 swap: values 0-3 stay in the lower
// row, 4-7 go to the upper), l <-> 15 - l (row_mirror, two independent
// chains), l <-> 7 - l (row_half_mirror), l ^ 2 and l ^ 1 (quad_perm).
__device__ __forceinline__ float reduce8h(float (&p)[8], int lane) {
#pragma unroll
  for (int k = 0; k < 4; ++k) { swap16(p[k], p[k + 4]); p[k] = p[k] + p[k + 4]; }
  const bool b3 = lane & 8, b2 = lane & 4;
  const float y0 = (b3 ? p[1] : p[0]) + dpp<0x140>(b3 ? p[0] : p[1]);  // value 4 b4 + b3
  const float y1 = (b3 ? p[3] : p[2]) + dpp<0x140>(b3 ? p[2] : p[3]);  // value 4 b4 + 2 + b3
  float z = (b2 ? y1 : y0) + dpp<0x141>(b2 ? y0 : y1);
  z = z + dpp<0x4E>(z);  // quad_perm [2,3,0,1]
  z = z + dpp<0xB1>(z);  // quad_perm [1,0,3,2]
  return z;
}
// Max and sum over the 32 lanes of each half-wave (bitwise the same in every
// lane of the half).
__device__ __forceinline__ float half_max(float x) {
  x = fmaxf(x, dpp<0xB1>(x));
  x = fmaxf(x, dpp<0x4E>(x));
  x = fmaxf(x, dpp<0x141>(x));
  x = fmaxf(x, dpp<0x140>(x));
  float y = x;
  swap16(x, y);
  return fmaxf(x, y);
}
__device__ __forceinline__ float half_sum(float x) {
  x = x + dpp<0xB1>(x);
  x = x + dpp<0x4E>(x);
  x = x + dpp<0x141>(x);
  x = x + dpp<0x140>(x);
  float y = x;
  swap16(x, y);
  return x + y;
}
// Both halves' values of v: a gets half 0's, b half 1's, in every lane.
__device__ __forceinline__ void halves_both(float v, float& a, float& b) {
  a = v;
  b = v;
  swap32(a, b);
}

// Chunks of 8 rows the folded layout holds for CPL columns per lane: 8 up to
// 128 columns, 6 beyond (the two-wave kernel runs a problem of more than 128
// columns on one wave only up to 6 chunks), at most 192 Kt registers.
__host__ __device__ constexpr int half_max_c8(int cpl) { return cpl <= 4 ? 8 : 6; }

// Iterations and outputs of one problem of c8 row chunks on this wave alone,
// in the folded layout; the caller has filled sAl and the first-update
// potentials Fl.  Gc [256] holds the column potentials by compact column, Sl
// [64][4] the demands of each lane's folded columns.
template <int CPL>
__device__ __forceinline__ void half_solve(const SkParams& p, int64_t pb, int32_t nh, int32_t nc, int c8,
                                           const int32_t* cpos, const int32_t* hpos, const int32_t* cidx,
                                           const int32_t* hidx, const float* sAl, float* Fl, float* ul, float* Gc,
                                           float* Sl, float kappa) {
  constexpr int MC = half_max_c8(CPL);  // chunks the registers hold; chunks q >= c8 are skipped
  constexpr int P = (CPL + 1) / 2;      // folded column pairs (c, c + P)
  const int lane = threadIdx.x & (kWave - 1);
  const int h = lane >> 5, cl = lane & 31;
  const int32_t R = p.R;
  const float* bd = p.b + pb * R;
  const float* Cb = p.C + pb * p.C_stride;
#define HV(c) (cl + 32 * (c) < nc)                 // column c of the lane exists
#define HJ(c) (HV(c) ? cidx[cl + 32 * (c)] : 0)   // its rank
#define FV(c) ((c) + P * h < CPL && cl + 32 * ((c) + P * h) < nc)  // folded column c of the lane exists
#define RV(q) (8 * (q) + (lane >> 3) < nh)        // the row the lane holds after reduce4
#define HR(q, r) (8 * (q) + 4 * h + (r))           // row r of chunk q in the lane's half
#define GL(c) Gc[cl + 32 * (c)]
  float* Sw = Sl + lane * 4;

  float K[4 * MC][CPL];
  float v[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    v[c] = HV(c) ? 1.f : 0.f;
    GL(c) = 0.f;  // both halves store the same value
  }
  // padding columns take demand 1, and padding rows supply 1 below, so that
  // their scalings come out as exactly 1 (in range, and Kt is 0 there)
#pragma unroll
  for (int c = 0; c < P; ++c) Sw[c] = FV(c) ? bd[cidx[cl + 32 * (c + P * h)]] : 1.f;
  auto demands = [&](float (&sB)[P]) {
#pragma unroll
    for (int c = 0; c < P; ++c) sB[c] = Sw[c];
  };
  // Kt of the lane's rows from the potentials (after the exact log-domain
  // update of each row's potential when row_update is set).  Rows past nh
  // take the cost row of row 0 and a zero Kt.
  auto build = [&](bool row_update) {
#pragma unroll
    for (int q = 0; q < MC; ++q) {
      if (q >= c8) break;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int gi = HR(q, r);
        const bool rv = gi < nh;
        const int gs = rv ? gi : 0;
        const float* crow = Cb + (int64_t)hidx[gs] * R;
        float cc[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) cc[c] = HV(c) ? crow[HJ(c)] * kappa : 0.f;
        float fi;
        if (row_update) {
          float t[CPL];
          float mx = -INFINITY;
#pragma unroll
          for (int c = 0; c < CPL; ++c) {
            t[c] = HV(c) ? (GL(c) + flog2(v[c])) - cc[c] : -INFINITY;
            mx = fmaxf(mx, t[c]);
          }
          mx = half_max(mx);
          float sum = 0.f;
#pragma unroll
          for (int c = 0; c < CPL; ++c) sum += HV(c) ? fexp2(t[c] - mx) : 0.f;
          sum = half_sum(sum);
          fi = flog2(sAl[gs]) - (mx + flog2(sum));
          if (rv && cl == 0) Fl[gi] = fi;
        } else {
          fi = Fl[gs];
        }
#pragma unroll
        for (int c = 0; c < CPL; ++c) K[4 * q + r][c] = rv && HV(c) ? fexp2((fi + GL(c)) - cc[c]) : 0.f;
      }
    }
  };

#define UST(q, val) \
  if ((lane & 7) == 0) ul[8 * (q) + (lane >> 3)] = (val)
#pragma unroll
  for (int q = 0; q < MC; ++q)
    if (q < c8) UST(q, RV(q) ? 1.f : 0.f);
  // Row half-steps take chunks in pairs (q, q + 1): reduce8h leaves the total
  // of row PR(q) in lane l; an odd last chunk goes through reduce4.
#define PR(q) (8 * ((q) + ((lane >> 4) & 1)) + 4 * h + 2 * ((lane >> 2) & 1) + ((lane >> 3) & 1))
  float sAp[MC / 2];
#pragma unroll
  for (int q = 0; q < MC; q += 2) sAp[q / 2] = PR(q) < nh ? sAl[PR(q)] : 1.f;
  const int qt = c8 - 1;  // the odd last chunk, when c8 is odd
  const float sAt = (c8 & 1) && RV(qt) ? sAl[8 * qt + (lane >> 3)] : 1.f;

  int32_t it = 1;
  bool skip_row = true;
  bool row_update = false;
  for (;;) {
    build(row_update);
    if (row_update) {
#pragma unroll
      for (int q = 0; q < MC; ++q)
        if (q < c8) UST(q, RV(q) ? 1.f : 0.f);
      row_update = false;
    }
    bool done = false, col_fail = false;
    for (;;) {
      if (!skip_row) {
        // ---- row half-step: u_i = s~_i / sum_c Kt_ic v_c ----------------------------
        uint32_t lo = 0xFFFFFFFFu, hi = 0u;
#pragma unroll
        for (int q = 0; q < MC; q += 2) {
          if (q >= c8) break;
          if (q + 1 < c8) {
            float pp[8];
#pragma unroll
            for (int r = 0; r < 8; ++r) {
              float acc = K[4 * q + r][0] * v[0];
#pragma unroll
              for (int c = 1; c < CPL; ++c) acc = __builtin_fmaf(K[4 * q + r][c], v[c], acc);
              pp[r] = acc;
            }
            const float y = reduce8h(pp, lane);  // all lanes take part
            const float un = sAp[q / 2] * frcp(PR(q) < nh ? y : 1.f);
            const uint32_t bits = __float_as_uint(un);
            lo = bits < lo ? bits : lo;
            hi = bits > hi ? bits : hi;
            if ((lane & 3) == 0) ul[PR(q)] = un;
          } else {
            float pp[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              float acc = K[4 * q + r][0] * v[0];
#pragma unroll
              for (int c = 1; c < CPL; ++c) acc = __builtin_fmaf(K[4 * q + r][c], v[c], acc);
              pp[r] = acc;
            }
            const float y = reduce4(pp, lane);
            const float un = sAt * frcp(RV(q) ? y : 1.f);
            const uint32_t bits = __float_as_uint(un);
            lo = bits < lo ? bits : lo;
            hi = bits > hi ? bits : hi;
            UST(q, un);
          }
        }
        const bool fail = !(lo >= __float_as_uint(kLo) && hi <= __float_as_uint(kHi));
        if (__ballot(fail) != 0) {
          row_update = true;
          skip_row = true;
          break;
        }
      }
      skip_row = false;
      // ---- column half-step: v_c = d_c / sum_i u_i Kt_ic --------------------------------
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      float x[CPL], x2[CPL];
#pragma unroll
      for (int c = 0; c < CPL; ++c) x[c] = x2[c] = 0.f;
      float4 ua = *reinterpret_cast<const float4*>(ul + 4 * h);
#pragma unroll
      for (int q = 0; q < MC; ++q) {
        if (q >= c8) break;
        float4 na = ua;  // the next chunk's scalings (past c8: unused)
        if (q + 1 < MC) na = *reinterpret_cast<const float4*>(ul + 8 * (q + 1) + 4 * h);
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          x[c] = __builtin_fmaf(ua.x, K[4 * q][c], x[c]);
          x2[c] = __builtin_fmaf(ua.y, K[4 * q + 1][c], x2[c]);
          x[c] = __builtin_fmaf(ua.z, K[4 * q + 2][c], x[c]);
          x2[c] = __builtin_fmaf(ua.w, K[4 * q + 3][c], x2[c]);
        }
        ua = na;
      }
      // fold: register c of half 0 gets column c, of half 1 column c + P
      float xf[P];
#pragma unroll
      for (int c = 0; c < P; ++c) {
        float a = x[c] + x2[c];
        float b = c + P < CPL ? x[c + P] + x2[c + P] : 0.f;
        swap32(a, b);
        xf[c] = a + b;
      }
      float sB[P];
      demands(sB);
      uint32_t clo = 0xFFFFFFFFu, chi = 0u;
#pragma unroll
      for (int c = 0; c < P; ++c) {
        const float vn = sB[c] * frcp(FV(c) ? xf[c] : 1.f);
        const uint32_t bits = __float_as_uint(vn);
        clo = bits < clo ? bits : clo;
        chi = bits > chi ? bits : chi;
        float a, b;
        halves_both(vn, a, b);
        v[c] = a;
        if (c + P < CPL) v[c + P] = b;
      }
      col_fail = __ballot(!(clo >= __float_as_uint(kLo) && chi <= __float_as_uint(kHi))) != 0;
      done = it == p.iters;
      if (!done) ++it;
      if (col_fail || done) break;
    }
    if (col_fail) {
      // exact log-domain update of every column (both halves alike), absorbed
      // into G; Kt is rebuilt at the top of the loop, or below after the last
      // iteration
      psync<1>();
      float mx[CPL], sum[CPL];
#pragma unroll
      for (int c = 0; c < CPL; ++c) { mx[c] = -INFINITY; sum[c] = 0.f; }
      for (int32_t i = 0; i < nh; ++i) {
        const float fi = Fl[i] + flog2(ul[i]);
        const float* crow = Cb + (int64_t)hidx[i] * R;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          if (HV(c)) {
            const float t = fi - crow[HJ(c)] * kappa;
            const float m2 = fmaxf(mx[c], t);
            sum[c] = sum[c] * fexp2(mx[c] - m2) + fexp2(t - m2);
            mx[c] = m2;
          }
        }
      }
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        GL(c) = HV(c) ? flog2(bd[HJ(c)]) - (mx[c] + flog2(sum[c])) : 0.f;
        v[c] = HV(c) ? 1.f : 0.f;
      }
      psync<1>();
      if (done) {
        build(false);
        break;
      }
      continue;
    }
    if (done) break;
  }

  // ---- plan, column cap, outputs -------------------------------------------------
  psync<1>();
  const bool colcap = !(p.flags & TAOT_SK_NO_COLCAP);
  float fac[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) fac[c] = 1.f;
  if (colcap) {
    float cs[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) cs[c] = 0.f;
#pragma unroll
    for (int q = 0; q < MC; ++q) {
      if (q >= c8) break;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float ui = ul[HR(q, r)];
#pragma unroll
        for (int c = 0; c < CPL; ++c) cs[c] += ui * K[4 * q + r][c] * v[c];
      }
    }
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      float a, b;
      halves_both(cs[c], a, b);
      const float tot = a + b;
      fac[c] = HV(c) ? fminf(1.f, bd[HJ(c)] / (tot + 1e-12f)) : 1.f;
    }
  }
  if (p.T) {
    float* Tb = p.T + pb * R * R;
    for (int32_t i = 0; i < R; ++i) {
      const bool hot = hpos[i] >= 0;
      for (int32_t j = lane; j < R; j += kWave)
        if (!hot || cpos[j] < 0) Tb[(int64_t)i * R + j] = 0.f;
    }
#pragma unroll
    for (int q = 0; q < MC; ++q) {
      if (q >= c8) break;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int gi = HR(q, r);
        if (gi < nh) {
          const float ui = ul[gi];
          float* trow = Tb + (int64_t)hidx[gi] * R;
#pragma unroll
          for (int c = 0; c < CPL; ++c)
            if (HV(c)) trow[HJ(c)] = ui * K[4 * q + r][c] * (v[c] * fac[c]);
        }
      }
    }
  }
  const float to_nat = p.eps * kLn2;
  for (int32_t i = lane; i < R; i += kWave) {
    const int32_t ih = hpos[i];
    if (p.f) p.f[pb * R + i] = ih >= 0 ? (Fl[ih] + flog2(ul[ih])) * to_nat : -INFINITY;
    if (p.g && cpos[i] < 0) p.g[pb * R + i] = -INFINITY;
  }
  if (p.g && h == 0) {
#pragma unroll
    for (int c = 0; c < CPL; ++c)
      if (HV(c)) p.g[pb * R + HJ(c)] = (GL(c) + flog2(v[c])) * to_nat;
  }
  if (lane == 0 && p.status) p.status[pb] = 0u;
#undef UST
#undef PR
#undef GL
#undef HR
#undef RV
#undef FV
#undef HJ
#undef HV
}

// The solver instance of wave wv (uniform over the wave).
template <int CPL, int C8W, int NW>
__device__ __forceinline__ void solve_on_wave(int wv, const SkParams& p, int64_t pb, int32_t nh, int32_t nc,
                                              const int32_t* cpos, const int32_t* hpos, const int32_t* cidx,
                                              const int32_t* hidx, const float* sAl, float* Fl, float* ul,
                                              float* Gall, float* Sall, float* xbuf, float kappa) {
  if constexpr (NW == 1) {
    wave_solve<CPL, C8W, 1, 0>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, kappa);
  } else if constexpr (NW == 2) {
    if (wv == 0) wave_solve<CPL, C8W, 2, 0>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, kappa);
    else wave_solve<CPL, C8W, 2, 1>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, kappa);
  } else {
    switch (wv) {
      case 0: wave_solve<CPL, C8W, 4, 0>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, kappa); break;
      case 1: wave_solve<CPL, C8W, 4, 1>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, kappa); break;
      case 2: wave_solve<CPL, C8W, 4, 2>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, kappa); break;
      default: wave_solve<CPL, C8W, 4, 3>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, kappa); break;
    }
  }
}

// One problem on NW waves (NW = 1: this wave alone, beside other one-wave
// problems of the workgroup; NW = W: the whole workgroup of the W-wave kernel).
template <int NW, int W>
__device__ __forceinline__ void wave_problem(const SkParams& p, int64_t pb, int32_t* wl) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = NW == 1 ? 0 : __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);  // uniform
  const int32_t R = p.R;
  // float arrays first: ul is read 16 bytes at a time
  float* sAl = reinterpret_cast<float*>(wl);  // [64] scaled supply
  float* Fl = sAl + 64;                       // [64] absorbed row potentials (log2 units)
  float* ul = Fl + 64;                        // [64] row scalings
  float* Gall = ul + 64;                      // [NW][4][64] column potentials
  float* Sall = Gall + NW * 4 * kWave;        // [NW][64][4] column demands
  float* xbuf = Sall + NW * 4 * kWave;        // [2][NW][4][64] column exchange (NW > 1)
  int32_t* iw = reinterpret_cast<int32_t*>(reinterpret_cast<float*>(wl) + wave_lds_floats(NW));
  int32_t* cpos = iw + 4;        // [R] compact column, -1 if not cold (iw[0..3] unused)
  int32_t* hpos = cpos + R;      // [R] compact row of rank i, -1 if not hot
  int32_t* cidx = hpos + R;      // [256]
  int32_t* hidx = cidx + 256;    // [64]
  const float* a = p.a + pb * R;
  const float* bd = p.b + pb * R;
  const float* Cb = p.C + pb * p.C_stride;

  // ---- supports and mass (every wave, identical results) --------------------
  double sa = 0.0, sd = 0.0;
  int32_t nh = 0, nc = 0;
  for (int32_t base = 0; base < R; base += kWave) {
    const int32_t i = base + lane;
    const bool in = i < R;
    const float ai = in ? a[i] : 0.f, bi = in ? bd[i] : 0.f;
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
  sa = wave_sum_d(sa);
  sd = wave_sum_d(sd);
  double gamma = __shfl(sd, 0, kWave) / fmax(__shfl(sa, 0, kWave), kEps0);
  gamma = gamma < 1.0 ? gamma : 1.0;
  sAl[lane] = lane < nh ? (float)(gamma * (double)a[hidx[lane]]) : 0.f;  // zero padding to 64 rows
  psync<NW>();
  const float kappa = kLog2e / p.eps;

  // ---- first row update over all R columns (v = 1): F_i = log2 s~_i - LSE2_j(-C'_ij),
  // rows dealt out over the waves (the class prepass has left problems with
  // a non-finite cost to the LDS or streamed kernel)
  for (int32_t i = wv; i < nh; i += NW) {
    const float* crow = Cb + (int64_t)hidx[i] * R;
    float mx = -INFINITY;
    for (int32_t j = lane; j < R; j += kWave) mx = fmaxf(mx, -crow[j] * kappa);
    mx = lanes_max(mx);
    float sum = 0.f;
    for (int32_t j = lane; j < R; j += kWave) sum += fexp2(-crow[j] * kappa - mx);
    sum = lanes_sum(sum);
    if (lane == 0) Fl[i] = flog2(sAl[i]) - (mx + flog2(sum));
  }
  psync<NW>();
  if constexpr (NW == 1 && W == 2) {
    // one wave alone: the folded layout (every single class of the two-wave
    // kernel fits it)
    const int cph = (nc + 31) / 32, c8 = (nh + 7) / 8;
    switch (cph) {
#define TAOT_HALF_CASE(CPL_)                                                                          \
  case CPL_:                                                                                          \
    if (c8 >= 1 && c8 <= half_max_c8(CPL_)) {                                                         \
      half_solve<CPL_>(p, pb, nh, nc, c8, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, kappa);    \
      return;                                                                                         \
    }                                                                                                 \
    break;
      TAOT_HALF_CASE(1) TAOT_HALF_CASE(2) TAOT_HALF_CASE(3) TAOT_HALF_CASE(4)
      TAOT_HALF_CASE(5) TAOT_HALF_CASE(6) TAOT_HALF_CASE(7) TAOT_HALF_CASE(8)
#undef TAOT_HALF_CASE
      default: break;
    }
  } else {
    const int cpl = nc <= 64 ? 1 : nc <= 128 ? 2 : 4;
    const int c8w = ((nh + 7) / 8 + NW - 1) / NW;
    switch (cpl * 16 + c8w) {
#define TAOT_WAVE_CASE(CPL_, C8W_)                                                                    \
  case CPL_ * 16 + C8W_:                                                                              \
    if constexpr (shape_ok(W, NW, CPL_, C8W_))                                                        \
      solve_on_wave<CPL_, C8W_, NW>(wv, p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, Gall, Sall, xbuf, \
                                    kappa);                                                           \
    break;
#define TAOT_WAVE_CPL(CPL_)                                                                           \
  TAOT_WAVE_CASE(CPL_, 1) TAOT_WAVE_CASE(CPL_, 2) TAOT_WAVE_CASE(CPL_, 3) TAOT_WAVE_CASE(CPL_, 4)      \
  TAOT_WAVE_CASE(CPL_, 5) TAOT_WAVE_CASE(CPL_, 6) TAOT_WAVE_CASE(CPL_, 7) TAOT_WAVE_CASE(CPL_, 8)
      TAOT_WAVE_CPL(1) TAOT_WAVE_CPL(2) TAOT_WAVE_CPL(4)
#undef TAOT_WAVE_CPL
#undef TAOT_WAVE_CASE
      default: break;
    }
  }
}

// LDS of one wave of a single item, rounded to 16 bytes.
__host__ __device__ constexpr size_t single_lds_bytes(int32_t R) { return (wave_lds_bytes(R, 1) + 15) / 16 * 16; }

// The register problems of a batch on workgroups of G waves (G = W, or G = 8
// for the two-wave shapes): item k < n_multi is multi[k] on waves 0 .. W-1
// (any further waves end at once, and a barrier only waits for the waves that
// have not ended); item n_multi + g holds G single problems, one per wave,
// each wave with its own LDS slice.
//
// Single group g pairs the heavier half of the list (dealt from its front)
// with the lighter half (from its back), G / 2 problems each.  With G = 8 the
// group is the whole compute unit (eight 256-VGPR waves, two per SIMD), and
// the waves that share a SIMD share its issue slots: each wave reads its SIMD
// from the HW_ID register, and the k-th heaviest problem of the group goes to
// the first wave of the k-th SIMD, the k-th lightest to its second wave, so
// that every SIMD carries about the same work.  Any placement still gives
// every wave one distinct slot (slots ordered by rank within the SIMD, then
// by SIMD).
template <int W, int G>
__global__ void __launch_bounds__(G * kWave, W == 4 ? 4 : 2)
sinkhorn_reg_kernel(SkParams p, const int32_t* __restrict__ multi, const int32_t* __restrict__ single,
                    const int32_t* __restrict__ counts) {
  extern __shared__ __attribute__((aligned(16))) int32_t wl[];
  __shared__ int32_t simd_of[G];
  const int32_t n_multi = counts[0], n_single = counts[1];
  const int32_t k = blockIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if (k < n_multi) {
    if (w < W) wave_problem<W, W>(p, multi[k], wl);
    return;
  }
  const int64_t g = k - n_multi, F = ((int64_t)n_single + 1) / 2;
  if (g * (G / 2) >= F) return;  // past the last group (uniform over the workgroup)
  int slot = w;
  if constexpr (G > W) {
    // HW_ID bits 5:4 hold the SIMD of the wave
    const int simd = (int)__builtin_amdgcn_s_getreg((1 << 11) | (4 << 6) | 4);
    if ((threadIdx.x & (kWave - 1)) == 0) simd_of[w] = simd;
    __syncthreads();
    auto rank = [&](int u) {
      int r = 0;
      for (int t = 0; t < u; ++t) r += simd_of[t] == simd_of[u];
      return r;
    };
    const int mr = rank(w);
    int pos = 0;
    for (int u = 0; u < G; ++u) {
      const int ru = rank(u);
      pos += ru < mr || (ru == mr && simd_of[u] < simd);
    }
    slot = __builtin_amdgcn_readfirstlane(pos);
  }
  const bool front = slot < G / 2;
  const int kk = front ? slot : slot - G / 2;
  const int64_t j = front ? g * (G / 2) + kk : (int64_t)n_single - 1 - (g * (G / 2) + kk);
  if (front ? j < F : (j >= F && j < n_single))
    wave_problem<1, W>(p, single[j], wl + (size_t)w * (single_lds_bytes(p.R) / 4));
}

// Register class of every problem (0: not a register problem).
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
  // invalid supplies, demands or costs: the LDS or streamed kernel reports them
  const bool any_bad = __ballot(bad) != 0 || cost_bad_wave(p, pb);
  int c = any_bad ? 0 : classify(nh, nc, p.flags);
  if (c == 0 && !any_bad) c = wide_class(nh, nc, p.flags);
  if (lane == 0) cls[pb] = c;
}

// Multi and single lists of the W-wave kernel (one block), each by descending
// per-wave work (ascending index within equal work), so that the workgroups
// dealt out in order start with the heaviest and mix heavy and light work on
// every compute unit; single groups join problems of similar work.
__global__ void __launch_bounds__(kSkThreads) wave_order_kernel(const int32_t* __restrict__ cls, int32_t B, int32_t W,
                                                                int32_t* __restrict__ multi,
                                                                int32_t* __restrict__ single,
                                                                int32_t* __restrict__ wide,
                                                                int32_t* __restrict__ counts) {
  __shared__ int32_t wave_cnt[kSkWaves];
  __shared__ unsigned long long present[2];  // multi / single: bit w if some problem has per-wave work w
  if (threadIdx.x == 0) present[0] = present[1] = 0ull;
  __syncthreads();
  for (int32_t b = threadIdx.x; b < B; b += kSkThreads) {
    const int32_t c = cls[b];
    if (!is_reg_class(c)) continue;
    const int cpl = class_cpl(c), c8 = class_c8(c);
    atomicOr(&present[is_single(W, cpl, c8) ? 1 : 0], 1ull << (c8_per_wave(W, cpl, c8) * cpl));
  }
  __syncthreads();
  for (int k = 0; k < 2; ++k) {
    const unsigned long long works = present[k];
    int32_t* list = k == 0 ? multi : single;
    int32_t n = 0;
    for (int32_t wk = 63; wk > 0; --wk) {
      if (!((works >> wk) & 1ull)) continue;
      for (int32_t base = 0; base < B; base += kSkThreads) {
        const int32_t b = base + (int32_t)threadIdx.x;
        const int32_t c = b < B ? cls[b] : 0;
        bool f = false;
        if (is_reg_class(c)) {
          const int cpl = class_cpl(c), c8 = class_c8(c);
          f = (is_single(W, cpl, c8) ? 1 : 0) == k && c8_per_wave(W, cpl, c8) * cpl == wk;
        }
        int32_t tot;
        const int32_t pos = chunk_compact(f, wave_cnt, tot);
        if (f) list[n + pos] = b;
        n += tot;
      }
    }
    if (threadIdx.x == 0) counts[k] = n;
  }
  // the wide problems, by index
  int32_t n = 0;
  for (int32_t base = 0; base < B; base += kSkThreads) {
    const int32_t b = base + (int32_t)threadIdx.x;
    const bool f = b < B && is_wide_class(cls[b]);
    int32_t tot;
    const int32_t pos = chunk_compact(f, wave_cnt, tot);
    if (f) wide[n + pos] = b;
    n += tot;
  }
  if (threadIdx.x == 0) counts[2] = n;
}

// ---------------------------------------------------------------------------
// Wide register path: problems with up to 96 hot ranks and up to 1024 cold
// ranks that the register classes do not take (large R).  One workgroup of
// 12 waves per problem keeps the whole |H| x |C| block of Kt in VGPRs: wave w
// holds rows 8w .. 8w+7, lane l the compact columns l + 64c (c < CPL).  The
// row half-step is wave-local, as in the register path.  The column
// half-step reduce-scatters the waves' partial sums through LDS: the owner of
// column slot c (wave c mod 12) adds the 12 partials in wave order and
// computes v for that slot, which every wave then reads back (two barriers
// per iteration).  Out-of-range scalings trigger the same exact log-domain
// updates.

// LDS of the wide kernel: floats sA, F, u [96], the partial column sums
// [12 waves][16 slots][64 lanes], v and G [16 slots][64 lanes]; then ints: flags [4], nh / nc
// [4], cpos, hpos [R], cidx [960], hidx [96].
__host__ __device__ constexpr size_t wide_lds_floats() {
  return (size_t)3 * kWideRows + (size_t)(kWideWaves + 2) * kWave * kWideMaxCpl;
}
__host__ __device__ constexpr size_t wide_lds_bytes(int32_t R) {
  return wide_lds_floats() * 4 + (size_t)(8 + 2 * R + kWideCols + kWideRows) * 4;
}

template <int CPL>
__device__ __forceinline__ void wide_solve(const SkParams& p, int64_t pb, int32_t nh, int32_t nc,
                                           const int32_t* cpos, const int32_t* hpos, const int32_t* cidx,
                                           const int32_t* hidx, const float* sAl, float* Fl, float* ul,
                                           float* part, float* vsh, float* gsh, int32_t* flag, float kappa) {
  constexpr int NO = (CPL + kWideWaves - 1) / kWideWaves;        // slots a wave owns, at most
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int rb = 8 * wv;
  const int32_t R = p.R;
  const float* bd = p.b + pb * R;
  const float* Cb = p.C + pb * p.C_stride;
#define CV(c) (lane + kWave * (c) < nc)
#define CJ(c) (CV(c) ? cidx[lane + kWave * (c)] : 0)
#define OWN(k) (wv + kWideWaves * (k) < CPL)
#define OC(k) (wv + kWideWaves * (k))
#define RV() (rb + (lane >> 3) < nh)
  // slot c of this lane in the [slot][lane] arrays (consecutive lanes, distinct banks)
  float* myv = vsh + lane;  // v, then the column-cap factors
  float* myg = gsh + lane;  // G
#define SLOT(c) ((c) * kWave)
  // v lives in LDS (vsh) and is read where it is needed, which keeps the
  // registers for the Kt block
  float K[8][CPL];
  float sBo[NO];  // demands of the slots this wave owns
#pragma unroll
  for (int k = 0; k < NO; ++k) {
    sBo[k] = (OWN(k) && CV(OC(k))) ? bd[CJ(OC(k))] : 0.f;
    if (OWN(k)) {
      myg[SLOT(OC(k))] = 0.f;
      myv[SLOT(OC(k))] = CV(OC(k)) ? 1.f : 0.f;
    }
  }
  if ((lane & 7) == 0) ul[rb + (lane >> 3)] = RV() ? 1.f : 0.f;
  const float sAq = sAl[rb + (lane >> 3)];
  __syncthreads();  // every G slot is set

  // Kt of this wave's rows from the potentials (optionally after the exact
  // log-domain update of the row potentials), as in the register path; the
  // costs are read again for Kt rather than kept, to bound the registers
  auto build = [&](bool row_update) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int gi = rb + i;
      if (gi < nh) {
        int32_t go = __builtin_amdgcn_readfirstlane(gi);
        asm volatile("" : "+s"(go));
        const float* crow = Cb + (int64_t)__builtin_amdgcn_readfirstlane(hidx[go]) * R;
        float fi;
        if (row_update) {
          float t[CPL];
          float mx = -INFINITY;
#pragma unroll
          for (int c = 0; c < CPL; ++c) {
            t[c] = CV(c) ? (myg[SLOT(c)] + flog2(myv[SLOT(c)])) - crow[CJ(c)] * kappa : -INFINITY;
            mx = fmaxf(mx, t[c]);
          }
          mx = lanes_max(mx);
          float sum = 0.f;
#pragma unroll
          for (int c = 0; c < CPL; ++c) sum += CV(c) ? fexp2(t[c] - mx) : 0.f;
          sum = lanes_sum(sum);
          fi = flog2(sAl[gi]) - (mx + flog2(sum));
          if (lane == 0) Fl[gi] = fi;
        } else {
          fi = Fl[gi];
        }
#pragma unroll
        for (int c = 0; c < CPL; ++c) K[i][c] = CV(c) ? fexp2((fi + myg[SLOT(c)]) - crow[CJ(c)] * kappa) : 0.f;
      } else {
#pragma unroll
        for (int c = 0; c < CPL; ++c) K[i][c] = 0.f;
      }
    }
  };

  int32_t it = 1;
  bool skip_row = true, row_update = false;
  for (;;) {
    build(row_update);
    if (row_update) {
      if ((lane & 7) == 0) ul[rb + (lane >> 3)] = RV() ? 1.f : 0.f;
      row_update = false;
    }
    bool done = false, col_fail = false;
    for (;;) {
      if (!skip_row) {
        // ---- row half-step on this wave's 8 rows ----------------------------------
        float v[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) v[c] = myv[SLOT(c)];
        float pp[8];
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          float acc = K[r][0] * v[0];
#pragma unroll
          for (int c = 1; c < CPL; ++c) acc = __builtin_fmaf(K[r][c], v[c], acc);
          pp[r] = acc;
        }
        const float y = reduce8(pp, lane);  // all lanes take part
        const bool rv = RV();
        const float un = sAq * frcp(rv ? y : 1.f);
        const uint32_t bits = __float_as_uint(rv ? un : 1.f);
        if ((lane & 7) == 0) ul[rb + (lane >> 3)] = un;
        if (__ballot(!(bits >= __float_as_uint(kLo) && bits <= __float_as_uint(kHi))) != 0) {
          row_update = true;
          skip_row = true;
          break;
        }
      }
      skip_row = false;
      // ---- column half-step: partial sums, reduce-scatter, v back to every wave ----
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      const float4 ua = *reinterpret_cast<const float4*>(ul + rb);
      const float4 ub = *reinterpret_cast<const float4*>(ul + rb + 4);
      const float us[8] = {ua.x, ua.y, ua.z, ua.w, ub.x, ub.y, ub.z, ub.w};
      {
        float x[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) x[c] = 0.f;
#pragma unroll
        for (int r = 0; r < 8; ++r)
#pragma unroll
          for (int c = 0; c < CPL; ++c) x[c] = __builtin_fmaf(us[r], K[r][c], x[c]);
        float* mine = part + wv * kWideMaxCpl * kWave + lane;
#pragma unroll
        for (int c = 0; c < CPL; ++c) mine[SLOT(c)] = x[c];
      }
      __syncthreads();
      uint32_t clo = 0xFFFFFFFFu, chi = 0u;
#pragma unroll
      for (int k = 0; k < NO; ++k) {
        if (OWN(k)) {
          const int c = OC(k);
          float s = part[SLOT(c) + lane];
#pragma unroll
          for (int w = 1; w < kWideWaves; ++w) s = s + part[w * kWideMaxCpl * kWave + SLOT(c) + lane];
          const float vn = sBo[k] * frcp(CV(c) ? s : 1.f);
          const uint32_t bits = __float_as_uint(CV(c) ? vn : 1.f);
          clo = bits < clo ? bits : clo;
          chi = bits > chi ? bits : chi;
          myv[SLOT(c)] = vn;
        }
      }
      if (__ballot(!(clo >= __float_as_uint(kLo) && chi <= __float_as_uint(kHi))) != 0 && lane == 0)
        atomicOr(&flag[1 + (it & 1)], 1);
      __syncthreads();
      col_fail = flag[1 + (it & 1)] != 0;  // the same on every wave
      if (threadIdx.x == 0) flag[1 + ((it + 1) & 1)] = 0;  // read by every wave before the barrier above
      done = it == p.iters;
      if (!done) ++it;
      if (col_fail || done) break;
    }
    if (col_fail) {
      // exact log-domain update of the owned columns (online LSE over all
      // rows), absorbed into G; Kt is rebuilt at the top of the loop
#pragma unroll
      for (int k = 0; k < NO; ++k) {
        if (OWN(k)) {
          const int c = OC(k);
          float mx = -INFINITY, sum = 0.f;
          if (CV(c)) {
            const int32_t j = cidx[lane + kWave * c];
            for (int32_t i = 0; i < nh; ++i) {
              const float t = (Fl[i] + flog2(ul[i])) - Cb[(int64_t)hidx[i] * R + j] * kappa;
              const float m2 = fmaxf(mx, t);
              sum = sum * fexp2(mx - m2) + fexp2(t - m2);
              mx = m2;
            }
          }
          myg[SLOT(c)] = CV(c) ? flog2(sBo[k]) - (mx + flog2(sum)) : 0.f;
          myv[SLOT(c)] = CV(c) ? 1.f : 0.f;
        }
      }
      __syncthreads();  // every G is set; every owner has read F and u
      if (done) {
        build(false);
        break;
      }
      continue;
    }
    if (done) break;
  }

  // ---- column cap, plan, potentials -----------------------------------------------
  __syncthreads();  // every wave's row scalings are in ul
  const float to_nat = p.eps * kLn2;
  float v[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) v[c] = myv[SLOT(c)];
  float fac[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) fac[c] = 1.f;
  if (!(p.flags & TAOT_SK_NO_COLCAP)) {
    {
      float cs[CPL];
#pragma unroll
      for (int c = 0; c < CPL; ++c) cs[c] = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float ui = ul[rb + i];
#pragma unroll
        for (int c = 0; c < CPL; ++c) cs[c] += ui * K[i][c] * v[c];
      }
      float* mine = part + wv * kWideMaxCpl * kWave + lane;
#pragma unroll
      for (int c = 0; c < CPL; ++c) mine[SLOT(c)] = cs[c];
    }
    __syncthreads();  // also: every wave has read v
#pragma unroll
    for (int k = 0; k < NO; ++k) {
      if (OWN(k)) {
        const int c = OC(k);
        float s = part[SLOT(c) + lane];
#pragma unroll
        for (int w = 1; w < kWideWaves; ++w) s = s + part[w * kWideMaxCpl * kWave + SLOT(c) + lane];
        myv[SLOT(c)] = CV(c) ? fminf(1.f, sBo[k] / (s + 1e-12f)) : 1.f;
      }
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < CPL; ++c) fac[c] = myv[SLOT(c)];
  }
  if (p.T) {
    float* Tb = p.T + pb * R * R;
    for (int32_t i = wv; i < R; i += kWideWaves) {
      const bool hot = hpos[i] >= 0;
      for (int32_t j = lane; j < R; j += kWave)
        if (!hot || cpos[j] < 0) Tb[(int64_t)i * R + j] = 0.f;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int gi = rb + i;
      if (gi < nh) {
        const float ui = ul[gi];
        float* trow = Tb + (int64_t)hidx[gi] * R;
#pragma unroll
        for (int c = 0; c < CPL; ++c)
          if (CV(c)) trow[CJ(c)] = ui * K[i][c] * (v[c] * fac[c]);
      }
    }
  }
  for (int32_t i = threadIdx.x; i < R; i += kWideThreads) {
    const int32_t ih = hpos[i];
    if (p.f) p.f[pb * R + i] = ih >= 0 ? (Fl[ih] + flog2(ul[ih])) * to_nat : -INFINITY;
    if (p.g && cpos[i] < 0) p.g[pb * R + i] = -INFINITY;
  }
  if (p.g) {
#pragma unroll
    for (int k = 0; k < NO; ++k)
      if (OWN(k) && CV(OC(k))) p.g[pb * R + CJ(OC(k))] = (myg[SLOT(OC(k))] + flog2(v[OC(k)])) * to_nat;
  }
  if (threadIdx.x == 0 && p.status) p.status[pb] = 0u;
#undef SLOT
#undef RV
#undef OC
#undef OWN
#undef CJ
#undef CV
}

// One wide problem on the 12 waves of a workgroup.
__device__ __forceinline__ void wide_problem(const SkParams& p, int64_t pb, int32_t* wl) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int32_t R = p.R;
  float* sAl = reinterpret_cast<float*>(wl);        // [96]
  float* Fl = sAl + kWideRows;                      // [96]
  float* ul = Fl + kWideRows;                       // [96]
  float* part = ul + kWideRows;                     // [12][16][64]
  float* vsh = part + kWideWaves * kWave * kWideMaxCpl;  // [16][64]
  float* gsh = vsh + kWave * kWideMaxCpl;           // [16][64]
  int32_t* iw = reinterpret_cast<int32_t*>(reinterpret_cast<float*>(wl) + wide_lds_floats());
  int32_t* flag = iw;        // [4]: flag[1 + parity] column failure of an iteration
  int32_t* cnt = iw + 4;     // [4]: nh, nc
  int32_t* cpos = iw + 8;    // [R]
  int32_t* hpos = cpos + R;  // [R]
  int32_t* cidx = hpos + R;  // [1024]
  int32_t* hidx = cidx + kWideCols;         // [96]
  const float* a = p.a + pb * R;
  const float* bd = p.b + pb * R;
  const float* Cb = p.C + pb * p.C_stride;

  // ---- supports and mass (wave 0) ---------------------------------------------
  if (wv == 0) {
    double sa = 0.0, sd = 0.0;
    int32_t nh = 0, nc = 0;
    for (int32_t base = 0; base < R; base += kWave) {
      const int32_t i = base + lane;
      const bool in = i < R;
      const float ai = in ? a[i] : 0.f, bi = in ? bd[i] : 0.f;
      sa += (double)ai;
      sd += (double)bi;
      const uint64_t hm = __ballot(in && ai > 0.f), cm = __ballot(in && bi > 0.f);
      const uint64_t below = (1ull << lane) - 1ull;
      const int32_t ph = nh + __popcll(hm & below), pc = nc + __popcll(cm & below);
      if (in) {
        hpos[i] = ai > 0.f ? ph : -1;
        cpos[i] = bi > 0.f ? pc : -1;
      }
      if (in && ai > 0.f && ph < kWideRows) hidx[ph] = i;
      if (in && bi > 0.f && pc < kWideCols) cidx[pc] = i;
      nh += __popcll(hm);
      nc += __popcll(cm);
    }
    sa = wave_sum_d(sa);
    sd = wave_sum_d(sd);
    double gamma = __shfl(sd, 0, kWave) / fmax(__shfl(sa, 0, kWave), kEps0);
    gamma = gamma < 1.0 ? gamma : 1.0;
    for (int32_t i = lane; i < kWideRows; i += kWave)
      sAl[i] = i < nh ? (float)(gamma * (double)a[hidx[i]]) : 0.f;  // zero padding
    if (lane == 0) {
      cnt[0] = nh;
      cnt[1] = nc;
      flag[0] = flag[1] = flag[2] = 0;
    }
  }
  __syncthreads();
  const int32_t nh = cnt[0], nc = cnt[1];
  const float kappa = kLog2e / p.eps;

  // ---- first row update over all R columns (v = 1), rows dealt out over the
  // waves (problems with a non-finite cost never reach this kernel)
  for (int32_t i = wv; i < nh; i += kWideWaves) {
    const float* crow = Cb + (int64_t)hidx[i] * R;
    float mx = -INFINITY;
    for (int32_t j = lane; j < R; j += kWave) mx = fmaxf(mx, -crow[j] * kappa);
    mx = lanes_max(mx);
    float sum = 0.f;
    for (int32_t j = lane; j < R; j += kWave) sum += fexp2(-crow[j] * kappa - mx);
    sum = lanes_sum(sum);
    if (lane == 0) Fl[i] = flog2(sAl[i]) - (mx + flog2(sum));
  }
  __syncthreads();
  switch (wide_cpl(nc)) {
#define TAOT_WIDE_CASE(CPL_)                                                                          \
  case CPL_:                                                                                          \
    wide_solve<CPL_>(p, pb, nh, nc, cpos, hpos, cidx, hidx, sAl, Fl, ul, part, vsh, gsh, flag, kappa); \
    break;
    TAOT_WIDE_CASE(4) TAOT_WIDE_CASE(6) TAOT_WIDE_CASE(8) TAOT_WIDE_CASE(10) TAOT_WIDE_CASE(12)
    TAOT_WIDE_CASE(14) TAOT_WIDE_CASE(15)
#undef TAOT_WIDE_CASE
    default: break;
  }
}

// The listed wide problems, a grid walking the list (one problem per
// workgroup at a time; the workgroup's LDS is reused by its next problem).
__global__ void __launch_bounds__(kWideThreads)
sinkhorn_wide_kernel(SkParams p, const int32_t* __restrict__ list, const int32_t* __restrict__ count) {
  extern __shared__ __attribute__((aligned(16))) int32_t wl[];
  const int32_t n = *count;
  for (int32_t k = blockIdx.x; k < n; k += gridDim.x) {
    wide_problem(p, list[k], wl);
    __syncthreads();
  }
}

template <int W, int G>
taot_status launch_reg_kernel(const SkParams& p, const int32_t* multi, const int32_t* single, const int32_t* counts,
                              hipStream_t stream) {
  const size_t lds = std::max(wave_lds_bytes(p.R, W), (size_t)G * single_lds_bytes(p.R));
  if (lds > 65536 && hipFuncSetAttribute((const void*)sinkhorn_reg_kernel<W, G>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return TAOT_ERR_LAUNCH;
  // one workgroup per item at most: B is an upper bound on the items
  hipLaunchKernelGGL((sinkhorn_reg_kernel<W, G>), dim3((unsigned)p.B), dim3(G * kWave), lds, stream, p, multi,
                     single, counts);
  return hipGetLastError() == hipSuccess ? TAOT_OK : TAOT_ERR_LAUNCH;
}

// The register path on the caller's stream: classes, lists, then one
// register kernel.  W = 4 when every problem can hold four 128-VGPR waves at
// once (four SIMDs per compute unit, four such waves per SIMD), else 2
// (TAOT_SK_WAVES_1 forces W = 2, i.e. one wave per problem where it fits).
taot_status launch_wave(const SkParams& p, int32_t* cls, int32_t* lists, int32_t* counts, hipStream_t stream) {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return TAOT_ERR_LAUNCH;
  const int64_t cap = (int64_t)cus * 4 * 4;
  const int W = (4 * (int64_t)p.B <= cap && !(p.flags & TAOT_SK_WAVES_1)) ? 4 : 2;
  hipLaunchKernelGGL(wave_class_kernel, dim3((unsigned)p.B), dim3(kWave), 0, stream, p, cls);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  int32_t* multi = lists;
  int32_t* single = lists + p.B;
  int32_t* wide = lists + 2 * (int64_t)p.B;
  hipLaunchKernelGGL(wave_order_kernel, dim3(1), dim3(kSkThreads), 0, stream, cls, p.B, W, multi, single, wide,
                     counts);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  // two-wave shapes run in eight-wave groups while their LDS slices fit 64 KB
  const bool g8 = 8 * single_lds_bytes(p.R) <= 65536;
  const taot_status st = W == 4 ? launch_reg_kernel<4, 4>(p, multi, single, counts, stream)
                         : g8   ? launch_reg_kernel<2, 8>(p, multi, single, counts, stream)
                                : launch_reg_kernel<2, 2>(p, multi, single, counts, stream);
  if (st != TAOT_OK) return st;
  // the wide problems: at most one workgroup per compute unit at a time
  const size_t lds = wide_lds_bytes(p.R);
  if (lds > 65536 && hipFuncSetAttribute((const void*)sinkhorn_wide_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                         (int)lds) != hipSuccess)
    return TAOT_ERR_LAUNCH;
  const unsigned grid = (unsigned)std::min<int64_t>(p.B, cus);
  hipLaunchKernelGGL(sinkhorn_wide_kernel, dim3(grid), dim3(kWideThreads), lds, stream, p, wide, counts + 2);
  return hipGetLastError() == hipSuccess ? TAOT_OK : TAOT_ERR_LAUNCH;
}

// Largest nh * nc over disjoint supports of R ranks (nh + nc <= R).
int64_t max_block(int32_t R) { return (int64_t)(R / 2) * (R - R / 2); }

struct SkWs {
  int32_t* flag;
  int32_t* cls;     // [B] register class
  int32_t* lists;   // [3][B] register problems: multi, single, wide
  int32_t* counts;  // [3]
  int32_t* cbad;    // [B or 1][scan_chunks(R)] chunk marks of the cost scan
  float* kt;
  int64_t kt_stride;
  size_t bytes;
};

SkWs carve(void* ws, int32_t B, int32_t R) {
  Carver c{static_cast<char*>(ws)};
  SkWs w;
  w.flag = c.take<int32_t>((size_t)B);
  w.cls = c.take<int32_t>((size_t)B);
  w.lists = c.take<int32_t>((size_t)3 * B);
  w.counts = c.take<int32_t>(3);
  w.cbad = c.take<int32_t>((size_t)B * scan_chunks(R));
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
  SkParams p{a, b, B, R, C, C_stride, eps, iters, flags, T, f, g, status, w.flag, w.kt, w.kt_stride, 0, 0,
             w.cbad, scan_chunks(R)};
  {
    const int64_t mats = C_stride ? B : 1;
    hipLaunchKernelGGL(cost_scan_kernel, dim3((unsigned)(mats * p.cchunks)), dim3(kScanThreads), 0, stream, C,
                       (int64_t)R * R, p.cchunks, w.cbad);
    if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  }
  const size_t vec_bytes = (size_t)kVecArrays * R * sizeof(float);
  const bool lds_path = R <= kLdsMaxR;
  if (!(flags & (TAOT_SK_FORCE_STREAM | TAOT_SK_NO_REGISTER))) {
    const taot_status st = launch_wave(p, w.cls, w.lists, w.counts, stream);
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
