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

#include "sk_common.h"

namespace taot {
namespace {

// Cost validation.  Every entry of a problem's C is checked (not only those
// the iterate reads): cost_scan_kernel marks each chunk of kScanChunk
// entries that holds a NaN or an infinity, once per call for a shared C and
// once per problem for per-problem costs; the class prepass and the LDS and
// streamed kernels OR the chunk marks of their problem's matrix.
// A chunk is 4096 entries: four 16-byte loads per thread of a 256-thread
// block, all in flight at once (a longer chunk per block leaves the scan
// waiting on one load after another).
constexpr int64_t kScanChunk = 4096;
constexpr int kScanThreads = 256;
constexpr int kScanLoads = 4;
static_assert(kScanChunk == 4 * kScanLoads * kScanThreads, "four float4 loads per thread and chunk");
__host__ __device__ constexpr int32_t scan_chunks(int32_t R) {
  return (int32_t)(((int64_t)R * R + kScanChunk - 1) / kScanChunk);
}

__global__ void __launch_bounds__(kScanThreads)
cost_scan_kernel(const float* __restrict__ C, int64_t R2, int32_t chunks, int32_t* __restrict__ cbad) {
  const int64_t mat = blockIdx.x / chunks, ch = blockIdx.x % chunks;
  const float* c = C + mat * R2;
  const int64_t lo = ch * kScanChunk, hi = lo + kScanChunk < R2 ? lo + kScanChunk : R2;
  int bad = 0;
  auto nonfinite = [](float x) { return (int)!(x - x == 0.f); };  // NaN or +-inf
  if (hi - lo == kScanChunk && (reinterpret_cast<uintptr_t>(c + lo) & 15u) == 0) {
    const float4* c4 = reinterpret_cast<const float4*>(c + lo) + threadIdx.x;
    float4 x[kScanLoads];
#pragma unroll
    for (int k = 0; k < kScanLoads; ++k) x[k] = c4[k * kScanThreads];
#pragma unroll
    for (int k = 0; k < kScanLoads; ++k)
      bad |= nonfinite(x[k].x) | nonfinite(x[k].y) | nonfinite(x[k].z) | nonfinite(x[k].w);
  } else {
    for (int64_t q = lo + threadIdx.x; q < hi; q += kScanThreads) bad |= nonfinite(c[q]);
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
// per-wave work, so that the workgroups dealt out in order start with the
// heaviest and mix heavy and light work on every compute unit; single groups
// join problems of similar work.  A counting sort over the per-wave work
// (below 64): count, exclusive scan from the heaviest down, place.  The order
// within equal work is whatever the atomics give: it changes the placement
// of problems on the chip, never a result.  Then the wide problems.
__global__ void __launch_bounds__(kSkThreads) wave_order_kernel(const int32_t* __restrict__ cls, int32_t B, int32_t W,
                                                                int32_t* __restrict__ multi,
                                                                int32_t* __restrict__ single,
                                                                int32_t* __restrict__ wide,
                                                                int32_t* __restrict__ counts) {
  __shared__ int32_t bins[3][64];  // multi, single, wide (bin 0) counts, then cursors
  for (int q = threadIdx.x; q < 3 * 64; q += kSkThreads) (&bins[0][0])[q] = 0;
  __syncthreads();
  auto key = [&](int32_t c, int& list) {
    if (is_wide_class(c)) { list = 2; return 0; }
    if (!is_reg_class(c)) { list = -1; return 0; }
    const int cpl = class_cpl(c), c8 = class_c8(c);
    list = is_single(W, cpl, c8) ? 1 : 0;
    return c8_per_wave(W, cpl, c8) * cpl;  // per-wave work, 1 .. 32
  };
  for (int32_t b = threadIdx.x; b < B; b += kSkThreads) {
    int list;
    const int wk = key(cls[b], list);
    if (list >= 0) atomicAdd(&bins[list][wk], 1);
  }
  __syncthreads();
  if (threadIdx.x < 3) {
    const int k = threadIdx.x;
    int32_t s = 0;
    for (int wk = 63; wk >= 0; --wk) {  // heaviest first
      const int32_t n = bins[k][wk];
      bins[k][wk] = s;
      s += n;
    }
    counts[k] = s;
  }
  __syncthreads();
  for (int32_t b = threadIdx.x; b < B; b += kSkThreads) {
    int list;
    const int wk = key(cls[b], list);
    if (list < 0) continue;
    const int32_t pos = atomicAdd(&bins[list][wk], 1);
    (list == 0 ? multi : list == 1 ? single : wide)[pos] = b;
  }
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
  const taot_status st = W == 4 ? launch_reg_w4g4(p, multi, single, counts, stream)
                         : g8   ? launch_reg_w2g8(p, multi, single, counts, stream)
                                : launch_reg_w2g2(p, multi, single, counts, stream);
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
  float* dn;        // [B][dn_stride] state of the dense streamed iterate
  int64_t dn_stride;
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
  w.dn_stride = round_up((int64_t)dense_state_floats(R), 64);
  w.dn = c.take<float>((size_t)B * w.dn_stride);
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
             w.cbad, scan_chunks(R), w.dn, w.dn_stride};
  {
    const int64_t mats = C_stride ? B : 1;
    hipLaunchKernelGGL(cost_scan_kernel, dim3((unsigned)(mats * p.cchunks)), dim3(kScanThreads), 0, stream, C,
                       (int64_t)R * R, p.cchunks, w.cbad);
    if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  }
  if (flags & (TAOT_SK_DENSE | TAOT_SK_LINEAR)) return launch_dense(p, stream);
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
