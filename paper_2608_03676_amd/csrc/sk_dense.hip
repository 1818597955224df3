// Dense streamed Sinkhorn (TAOT_SK_DENSE): the iterate of Sec. A.2 over all
// R x R entries of every problem, without the support compaction of the
// other paths (rows with no supply and columns with no demand are swept too
// and contribute nothing), in the GEMV form the paper writes the iteration
// in: u = s~ / (K v), v = d / (K^T u).
//
// Stabilisation is that of the other paths.  In log2 units (C' = C log2(e) /
// eps) the potentials F, G absorb the scalings whenever one leaves
// [2^-60, 2^60], and K~_ij = exp2(F_i + G_j - C'_ij) is kept in the
// workspace (one R x R matrix per problem); the iterations update only the
// scalings u, v, so their rounding stays relative.  The first row update is
// the exact log-domain one over all R columns from G = 0 (v = 1); an
// out-of-range scaling triggers the exact log-domain update of its row or
// column from C, with its row or column of K~ rebuilt.
//
// Each iteration is two grid-wide kernels over all problems, which keeps
// every compute unit streaming K~ from device memory:
//   row pass (B * R / 64 blocks of 64 rows): the rows' sums (K~ v)_i, u_i,
//       and the u-weighted column sums of the same rows, from registers, so
//       K~ is read once per iteration; the block writes its column partials
//       once.  dense_roww_kernel (R % 4 == 0): each wave streams 16 rows
//       with the next rows in flight; dense_row_kernel (other R): phases of
//       rows shared by the block's four waves.  (The first iteration builds
//       K~ instead, from the exact first row update.)
//   dense_col_kernel (B * R / 16 blocks): sums the blocks' partials of a
//       column in a fixed order and sets v_j.
// All reductions run in a fixed order, so results do not depend on
// scheduling.
#include <type_traits>

#include "sk_common.h"

namespace taot {
namespace {

constexpr int kDnThreads = 256;
constexpr int kDnWaves = kDnThreads / kWave;
constexpr int kDnRowBlock = 64;  // rows per block of the row pass
constexpr int kDnColBlock = 16;  // columns per block of the column kernel
constexpr int kDnDepth = 1;      // row tiles in flight behind the current one

// Row pass, R % 4 == 0 and C 16-byte aligned: the wave-streamed kernel, 16
// rows per wave, lane l holding the 16-byte groups l + 64 k (k < KQ) of a
// row.  Otherwise the phased kernel: thread t owns KPT columns t + 256 s, a
// phase holds TR rows of them in registers (TR * KPT <= 32) with the next
// phase's rows in flight.  Either way a block takes 64 rows.
constexpr int kDnWaveRows = kDnRowBlock / kDnWaves;
__host__ __device__ constexpr int pow2_at_least(int32_t x) { return x <= 1 ? 1 : x <= 2 ? 2 : x <= 4 ? 4 : 8; }
__host__ __device__ constexpr int dense_kq(int32_t R) { return pow2_at_least((R / 4 + kWave - 1) / kWave); }
__host__ __device__ constexpr int dense_kpt(int32_t R) { return pow2_at_least((R + kDnThreads - 1) / kDnThreads); }
__host__ __device__ constexpr int dense_tr_nc(int nc) { return 32 / nc < 8 ? 32 / nc : 8; }
__host__ __device__ constexpr int32_t dense_blocks(int32_t R) { return (R + kDnRowBlock - 1) / kDnRowBlock; }
__host__ __device__ constexpr int ilog2c(int x) { return x <= 1 ? 0 : 1 + ilog2c(x / 2); }

// Per-problem state (floats): F, G, u, v, s~ [R], then the column partials
// [row blocks][R].  K~ is the streamed-plan storage of the workspace.
struct DenseState {
  float* F;
  float* G;
  float* u;
  float* v;
  float* sA;
  float* part;
  float* K;
};
__device__ __forceinline__ DenseState dense_state(const SkParams& p, int64_t pb) {
  const int32_t R = p.R;
  float* s = p.dn_ws + pb * p.dn_stride;
  return {s, s + R, s + 2 * R, s + 3 * R, s + 4 * R, s + 5 * R, p.kt_ws + pb * p.kt_stride};
}

__device__ __forceinline__ bool in_range(float x) { return x >= kLo && x <= kHi; }

__device__ __forceinline__ bool cost_bad_block(const SkParams& p, int64_t pb) {
  const int64_t base = (p.C_stride ? pb : 0) * p.cchunks;
  bool bad = false;
  for (int32_t k = threadIdx.x; k < p.cchunks; k += kDnThreads) bad |= p.cbad[base + k] != 0;
  return __syncthreads_or(bad) != 0;
}

// Validation, supply scaling and the start (G = 0, v = 1 on all R columns),
// one block per problem.  A problem with bad input or no mass is finished
// here (T = 0, f = g = -inf, status) and skipped by the later kernels
// (stream_flag holds its status).
__global__ void __launch_bounds__(kDnThreads) dense_init_kernel(SkParams p) {
  __shared__ double red[2][kDnWaves];
  __shared__ int32_t cnt[2][kDnWaves];
  const int64_t pb = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
  const int32_t R = p.R;
  const float* a = p.a + pb * R;
  const float* bd = p.b + pb * R;
  const DenseState S = dense_state(p, pb);
  bool bad = false;
  double sa = 0.0, sd = 0.0;
  int32_t nh = 0, nc = 0;
  for (int32_t i = tid; i < R; i += kDnThreads) {
    const float ai = a[i], bi = bd[i];
    bad |= !(ai >= 0.f && ai <= 3.402823466e38f) || !(bi >= 0.f && bi <= 3.402823466e38f);
    sa += (double)ai;
    sd += (double)bi;
    nh += ai > 0.f;
    nc += bi > 0.f;
  }
  const bool cost_bad = cost_bad_block(p, pb);
  bad = __syncthreads_or(bad) != 0 || cost_bad;
  sa = wave_sum_d(sa);
  sd = wave_sum_d(sd);
  nh = (int32_t)wave_sum_i64(nh);
  nc = (int32_t)wave_sum_i64(nc);
  if (lane == 0) { red[0][wid] = sa; red[1][wid] = sd; cnt[0][wid] = nh; cnt[1][wid] = nc; }
  __syncthreads();
  double Sa = 0.0, Sd = 0.0;
  int32_t Nh = 0, Nc = 0;
  for (int w = 0; w < kDnWaves; ++w) { Sa += red[0][w]; Sd += red[1][w]; Nh += cnt[0][w]; Nc += cnt[1][w]; }
  double gamma = Sd / (Sa > kEps0 ? Sa : kEps0);
  gamma = gamma < 1.0 ? gamma : 1.0;
  const uint32_t st = bad ? TAOT_ST_BAD_INPUT : (Nh == 0 || Nc == 0) ? TAOT_ST_ZERO_MASS : 0u;
  if (tid == 0) p.stream_flag[pb] = (int32_t)st;
  if (st) {
    if (p.T)
      for (int64_t q = tid; q < (int64_t)R * R; q += kDnThreads) p.T[pb * R * R + q] = 0.f;
    for (int32_t i = tid; i < R; i += kDnThreads) {
      if (p.f) p.f[pb * R + i] = -INFINITY;
      if (p.g) p.g[pb * R + i] = -INFINITY;
    }
    if (tid == 0 && p.status) p.status[pb] = st;
    return;
  }
  for (int32_t i = tid; i < R; i += kDnThreads) {
    const float ai = a[i];
    S.sA[i] = ai > 0.f ? (float)(gamma * (double)ai) : 0.f;
    S.G[i] = 0.f;
    S.v[i] = 1.f;
  }
}

// Transposed butterfly reduce-scatter of N values per lane over the wave
// (N a power of two up to 64): N / 2 exchanges halve the vector at each of the
// masks 32, 16, ..., 64 / N, then a full butterfly over the remaining lane
// bits.  Lane l returns the wave total of value (l >> (6 - log2 N)) & (N - 1);
// the order of the additions is fixed, so every lane holding a total holds
// the same bits.
template <int N, typename Op>
__device__ __forceinline__ float wave_reduce_scatter(float (&v)[N], Op op) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int h = N / 2, m = 32; h >= 1; h /= 2, m /= 2) {
    const bool up = (lane & m) != 0;
#pragma unroll
    for (int k = 0; k < h; ++k) {
      const float send = up ? v[k] : v[k + h];
      const float keep = up ? v[k + h] : v[k];
      v[k] = op(keep, __shfl_xor(send, m, kWave));
    }
  }
  float x = v[0];
#pragma unroll
  for (int m = 32 / N; m > 0; m /= 2) x = op(x, __shfl_xor(x, m, kWave));
  return x;
}
struct OpAdd {
  __device__ float operator()(float a, float b) const { return a + b; }
};
struct OpMax {
  __device__ float operator()(float a, float b) const { return fmaxf(a, b); }
};

// Calls f(integral_constant<int, k>) for k = 0 .. N-1 in order.
template <int N>
struct Unrolled {
  template <typename F>
  __device__ __forceinline__ static void run(F& f) {
    Unrolled<N - 1>::run(f);
    f(std::integral_constant<int, N - 1>{});
  }
};
template <>
struct Unrolled<0> {
  template <typename F>
  __device__ __forceinline__ static void run(F&) {}
};

// Loads rows [0, nr) of the R-wide matrix at src into the thread's columns of
// t (zeros for rows >= nr and columns >= R).
template <int VEC, int KPT, int TR>
__device__ __forceinline__ void load_tile(const float* src, int32_t R, int32_t nr, float (&t)[TR][VEC * KPT]) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int r = 0; r < TR; ++r)
#pragma unroll
    for (int s = 0; s < KPT; ++s) {
      const int32_t q = tid + kDnThreads * s;
      if (VEC == 4) {
        float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
        if (r < nr && 4 * q < R) x = *reinterpret_cast<const float4*>(src + (int64_t)r * R + 4 * q);
        t[r][4 * s] = x.x;
        t[r][4 * s + 1] = x.y;
        t[r][4 * s + 2] = x.z;
        t[r][4 * s + 3] = x.w;
      } else {
        t[r][s] = r < nr && q < R ? src[(int64_t)r * R + q] : 0.f;
      }
    }
}

// Stores the thread's columns of one row.
template <int VEC, int KPT>
__device__ __forceinline__ void store_row(float* dst, int32_t R, const float (&x)[VEC * KPT]) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int s = 0; s < KPT; ++s) {
    const int32_t q = tid + kDnThreads * s;
    if (VEC == 4) {
      if (4 * q < R)
        *reinterpret_cast<float4*>(dst + 4 * q) = make_float4(x[4 * s], x[4 * s + 1], x[4 * s + 2], x[4 * s + 3]);
    } else if (q < R) {
      dst[q] = x[s];
    }
  }
}

// Column index of the thread's value c (VEC * KPT of them).
template <int VEC>
__device__ __forceinline__ int32_t col_of(int c) {
  return VEC == 4 ? 4 * ((int)threadIdx.x + kDnThreads * (c / 4)) + (c & 3) : (int)threadIdx.x + kDnThreads * c;
}

// One row half-step of the problem's row block: per phase of TR rows, the
// partial products K~_ic v_c of the thread's columns, a transposed reduction
// over the wave and the four waves' totals in LDS give every thread all TR
// sums (in a fixed order), hence u_i = s~_i / (K~ v)_i; then the u-weighted
// column sums of the thread's columns.  A row whose u_i leaves [2^-60, 2^60]
// takes the exact log-domain update from C (F_i absorbs it, u_i = 1) with its
// row of K~ rebuilt.  With BUILD (the first iteration) the tiles are of C and
// every row with supply takes the exact update from G = 0, v = 1, which
// builds K~.  The block writes its column partials once.
template <int VEC, int KPT, bool BUILD>
__global__ void __launch_bounds__(kDnThreads) __attribute__((amdgpu_waves_per_eu(BUILD || VEC * KPT > 4 ? 1 : 4))) dense_row_kernel(SkParams p, float kappa) {
  constexpr int NC = VEC * KPT, TR = dense_tr_nc(NC), PH = kDnRowBlock / TR, RB = kDnRowBlock, LG = ilog2c(TR);
  __shared__ float4 red[2][2][TR];         // [phase parity][max, sum][row] per-wave totals
  __shared__ float fixr[2][kDnWaves];      // per-wave max / sum of a fixed row
  __shared__ float sal[RB];
  const int32_t R = p.R, NB = (R + RB - 1) / RB;
  const int64_t pb = blockIdx.x / NB;
  const int32_t blk = blockIdx.x % NB;
  if (p.stream_flag[pb] != 0) return;  // uniform per block
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
  const DenseState S = dense_state(p, pb);
  const float* Cb = p.C + pb * p.C_stride;
  const int32_t r0 = blk * RB;
  const bool linear = (p.flags & TAOT_SK_LINEAR) != 0;
  for (int32_t r = tid; r < RB; r += kDnThreads) sal[r] = r0 + r < R ? S.sA[r0 + r] : 0.f;
  // G_c, v_c and G_c + log2 v_c of the thread's columns (-inf off the matrix
  // and where v_c = 0)
  float Gc[NC], vc[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int32_t j = col_of<VEC>(c);
    Gc[c] = j < R ? S.G[j] : -INFINITY;
    vc[c] = j < R ? S.v[j] : 0.f;
  }
  auto lv = [&](int c) { return vc[c] > 0.f ? Gc[c] + flog2(vc[c]) : -INFINITY; };
  float cs[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) cs[c] = 0.f;
  const float* src = BUILD ? Cb : S.K;
  // tiles of the next kDnDepth phases in flight behind the current one
  float buf[kDnDepth + 1][TR][NC];
#pragma unroll
  for (int d = 0; d < kDnDepth; ++d)
    if (r0 + d * TR < R)
      load_tile<VEC, KPT, TR>(src + (int64_t)(r0 + d * TR) * R, R, R - r0 - d * TR < TR ? R - r0 - d * TR : TR,
                              buf[d]);
  __syncthreads();  // sal
  const int wr = (lane >> (6 - LG)) & (TR - 1);       // the row whose wave total this lane holds
  const bool writer = (lane & ((kWave >> LG) - 1)) == 0;
  // the phases, unrolled at compile time (the tile buffers stay in registers)
  auto phase = [&](auto phc) __attribute__((always_inline)) {
    constexpr int ph = decltype(phc)::value;
    const int32_t i0 = r0 + ph * TR;
    if (i0 >= R) return;  // uniform
    const int32_t nr = R - i0 < TR ? R - i0 : TR;
    const int32_t ia = i0 + kDnDepth * TR;  // first row of the phase to issue
    if (ph + kDnDepth < PH && ia < R)
      load_tile<VEC, KPT, TR>(src + (int64_t)ia * R, R, R - ia < TR ? R - ia : TR, buf[(ph + kDnDepth) % (kDnDepth + 1)]);
    float (&cur)[TR][NC] = buf[ph % (kDnDepth + 1)];
    const int par = ph & 1;
    float uo = 0.f;  // u_i of row i0 + tid (tid < TR)
    if (BUILD && !linear) {
      // exact first row update: x_ic = (G_c + log2 v_c) - C'_ic
      float pm[TR];
#pragma unroll
      for (int r = 0; r < TR; ++r) {
        pm[r] = -INFINITY;
#pragma unroll
        for (int c = 0; c < NC; ++c) pm[r] = fmaxf(pm[r], lv(c) - cur[r][c] * kappa);
      }
      const float mw = wave_reduce_scatter<TR>(pm, OpMax());
      if (writer) reinterpret_cast<float*>(&red[par][0][wr])[wid] = mw;
      __syncthreads();
      float M[TR], ps[TR];
#pragma unroll
      for (int r = 0; r < TR; ++r) {
        const float4 w = red[par][0][r];
        M[r] = fmaxf(fmaxf(fmaxf(w.x, w.y), w.z), w.w);
        ps[r] = 0.f;
#pragma unroll
        for (int c = 0; c < NC; ++c)
          if (vc[c] > 0.f) ps[r] += fexp2((lv(c) - cur[r][c] * kappa) - M[r]);
      }
      const float sw = wave_reduce_scatter<TR>(ps, OpAdd());
      if (writer) reinterpret_cast<float*>(&red[par][1][wr])[wid] = sw;
      __syncthreads();
#pragma unroll
      for (int r = 0; r < TR; ++r) {
        if (r >= nr) break;
        const float4 w = red[par][1][r];
        const float sa = sal[ph * TR + r];
        const float fi = sa > 0.f ? flog2(sa) - (M[r] + flog2(((w.x + w.y) + w.z) + w.w)) : -INFINITY;
        float k[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          k[c] = sa > 0.f && Gc[c] != -INFINITY ? fexp2((fi + Gc[c]) - cur[r][c] * kappa) : 0.f;
          cs[c] += k[c];
        }
        store_row<VEC, KPT>(S.K + (int64_t)(i0 + r) * R, R, k);
        if (tid == r) {
          S.F[i0 + r] = fi;
          uo = sa > 0.f ? 1.f : 0.f;
        }
      }
    } else {
      if (BUILD) {
        // linear domain: M_ij = exp(-C_ij / eps) = exp2(-C'_ij), stored once
#pragma unroll
        for (int r = 0; r < TR; ++r) {
#pragma unroll
          for (int c = 0; c < NC; ++c) cur[r][c] = r < nr && col_of<VEC>(c) < R ? fexp2(-(cur[r][c] * kappa)) : 0.f;
          if (r < nr) store_row<VEC, KPT>(S.K + (int64_t)(i0 + r) * R, R, cur[r]);
        }
        if (tid < nr) S.F[i0 + tid] = 0.f;
      }
      float py[TR];
#pragma unroll
      for (int r = 0; r < TR; ++r) {
        py[r] = 0.f;
#pragma unroll
        for (int c = 0; c < NC; ++c) py[r] = __builtin_fmaf(cur[r][c], vc[c], py[r]);
      }
      const float yw = wave_reduce_scatter<TR>(py, OpAdd());
      if (writer) reinterpret_cast<float*>(&red[par][0][wr])[wid] = yw;
      __syncthreads();
      float u[TR];
      uint32_t bad = 0;
#pragma unroll
      for (int r = 0; r < TR; ++r) {
        const float4 w = red[par][0][r];
        const float sa = sal[ph * TR + r];
        u[r] = sa > 0.f ? sa * frcp(((w.x + w.y) + w.z) + w.w) : 0.f;
        if (!linear && sa > 0.f && !in_range(u[r])) bad |= 1u << r;
      }
      // rows out of range: exact log-domain update from C, one row at a time
      for (uint32_t m = bad; m; m &= m - 1) {
        const int r = __builtin_ctz(m);
        const int32_t i = i0 + r;
        float cr[NC], x[NC];
        const float* crow = Cb + (int64_t)i * R;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          const int32_t j = col_of<VEC>(c);
          cr[c] = j < R ? crow[j] : 0.f;
        }
        float mx = -INFINITY;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          x[c] = vc[c] > 0.f ? lv(c) - cr[c] * kappa : -INFINITY;
          mx = fmaxf(mx, x[c]);
        }
        mx = wave_max(mx);
        if (lane == 0) fixr[0][wid] = mx;
        __syncthreads();
        const float M = fmaxf(fmaxf(fmaxf(fixr[0][0], fixr[0][1]), fixr[0][2]), fixr[0][3]);
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < NC; ++c)
          if (x[c] != -INFINITY) s += fexp2(x[c] - M);
        s = wave_sum(s);
        if (lane == 0) fixr[1][wid] = s;
        __syncthreads();
        const float fi = flog2(sal[ph * TR + r]) - (M + flog2(((fixr[1][0] + fixr[1][1]) + fixr[1][2]) + fixr[1][3]));
        float k[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          k[c] = Gc[c] != -INFINITY ? fexp2((fi + Gc[c]) - cr[c] * kappa) : 0.f;
          cs[c] += k[c];
        }
        store_row<VEC, KPT>(S.K + (int64_t)i * R, R, k);
        if (tid == 0) S.F[i] = fi;
      }
#pragma unroll
      for (int r = 0; r < TR; ++r) {
        const float ur = (bad >> r) & 1u ? 0.f : u[r];
#pragma unroll
        for (int c = 0; c < NC; ++c) cs[c] = __builtin_fmaf(ur, cur[r][c], cs[c]);
        if (tid == r) uo = (bad >> r) & 1u ? 1.f : u[r];
      }
    }
    if (tid < nr) S.u[i0 + tid] = uo;
  };
  Unrolled<PH>::run(phase);
  store_row<VEC, KPT>(S.part + (int64_t)blk * R, R, cs);
}

// Loads one row's 16-byte groups of lane l (l + 64 k, k < KQ; zeros past R).
template <int KQ>
__device__ __forceinline__ void load_row4(const float* row, int32_t R, float (&x)[4 * KQ]) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int k = 0; k < KQ; ++k) {
    const int32_t q = lane + kWave * k;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (4 * q < R) v = reinterpret_cast<const float4*>(row)[q];
    x[4 * k] = v.x;
    x[4 * k + 1] = v.y;
    x[4 * k + 2] = v.z;
    x[4 * k + 3] = v.w;
  }
}
template <int KQ>
__device__ __forceinline__ void store_row4(float* row, int32_t R, const float (&x)[4 * KQ]) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int k = 0; k < KQ; ++k) {
    const int32_t q = lane + kWave * k;
    if (4 * q < R) reinterpret_cast<float4*>(row)[q] = make_float4(x[4 * k], x[4 * k + 1], x[4 * k + 2], x[4 * k + 3]);
  }
}

// Exact log-domain update of one row on this wave: c holds the row of C on
// entry (lane's columns), K~'s new row on exit; returns F_i.
// F_i = log2 s~_i - LSE2_j (G_j + log2 v_j - C'_ij) over the columns with
// v_j > 0, K~_ij = exp2(F_i + G_j - C'_ij) (0 where G_j = -inf).
template <int NC>
__device__ __forceinline__ float row_exact4(float (&c)[NC], const float (&G)[NC], const float (&vc)[NC], float sa,
                                            float kappa) {
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < NC; ++j)
    if (vc[j] > 0.f) mx = fmaxf(mx, (G[j] + flog2(vc[j])) - c[j] * kappa);
  mx = lanes_max(mx);
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < NC; ++j)
    if (vc[j] > 0.f) sum += fexp2(((G[j] + flog2(vc[j])) - c[j] * kappa) - mx);
  sum = lanes_sum(sum);
  const float fi = flog2(sa) - (mx + flog2(sum));
#pragma unroll
  for (int j = 0; j < NC; ++j) c[j] = G[j] != -INFINITY ? fexp2((fi + G[j]) - c[j] * kappa) : 0.f;
  return fi;
}

// Row half-step for R % 4 == 0, wave-streamed: each wave takes 16 rows of
// its block's 64, one at a time with the next P - 1 rows in flight (P rows
// of registers).  A row's sum (K~ v)_i is a fixed-order fold of the lane's
// products and then a butterfly over the wave (every lane gets the same
// bits), so every lane derives u_i = s~_i / (K~ v)_i and adds u_i K~_ij into
// its column sums.  An out-of-range u_i takes the exact log-domain update
// from the row of C in place.  With BUILD (the first iteration) the rows are
// of C and every row with supply takes the exact update from G = 0, v = 1,
// which writes K~.  The block's four waves add their column sums in LDS in
// wave order and write the block's partials once.
template <int KQ, bool BUILD>
__global__ void __launch_bounds__(kDnThreads) __attribute__((amdgpu_waves_per_eu(BUILD || KQ > 4 ? 1 : 4)))
dense_roww_kernel(SkParams p, float kappa) {
  constexpr int NC = 4 * KQ;
  constexpr int P = 64 / NC < 8 ? 64 / NC : 8;  // rows of the ring
  extern __shared__ __attribute__((aligned(16))) float wpart[];  // [kDnWaves][R] the waves' column sums
  const int32_t R = p.R, RB = kDnRowBlock, NB = dense_blocks(R);
  const int64_t pb = blockIdx.x / NB;
  const int32_t blk = blockIdx.x % NB;
  if (p.stream_flag[pb] != 0) return;  // uniform per block
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
  const DenseState S = dense_state(p, pb);
  const float* Cb = p.C + pb * p.C_stride;
  const int32_t r0 = blk * RB + wid * kDnWaveRows;
  const int32_t nrows = R - r0 <= 0 ? 0 : (R - r0 < kDnWaveRows ? R - r0 : kDnWaveRows);
  const bool linear = (p.flags & TAOT_SK_LINEAR) != 0;
  const float* src = BUILD ? Cb : S.K;
  float buf[P][NC];
#pragma unroll
  for (int d = 0; d + 1 < P; ++d)
    if (d < nrows) load_row4<KQ>(src + (int64_t)(r0 + d) * R, R, buf[d]);
  float vc[NC];
  load_row4<KQ>(S.v, R, vc);
  const float sal = lane < nrows ? S.sA[r0 + lane] : 0.f;  // lane k: the supply of row r0 + k
  float cs[NC];
#pragma unroll
  for (int j = 0; j < NC; ++j) cs[j] = 0.f;
  float uo = 0.f;  // lane k: u of row r0 + k
  uint32_t bad = 0;  // rows whose u left [2^-60, 2^60] (the same on every lane)
  auto row = [&](auto kc) __attribute__((always_inline)) {
    constexpr int k = decltype(kc)::value;
    if (k >= nrows) return;  // uniform
    if (k + P - 1 < nrows) load_row4<KQ>(src + (int64_t)(r0 + k + P - 1) * R, R, buf[(k + P - 1) % P]);
    float (&x)[NC] = buf[k % P];
    const int32_t i = r0 + k;
    const float sa = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sal), k));
    float u = 0.f;
    bool step = !BUILD;  // the row takes the scaling update from its row of K~
    if (BUILD && linear) {
      // M_ij = exp(-C_ij / eps) = exp2(-C'_ij), stored once
#pragma unroll
      for (int j = 0; j < NC; ++j) {
        const int32_t col = 4 * (lane + kWave * (j / 4)) + (j & 3);
        x[j] = col < R ? fexp2(-(x[j] * kappa)) : 0.f;
      }
      store_row4<KQ>(S.K + (int64_t)i * R, R, x);
      if (lane == 0) S.F[i] = 0.f;
      step = true;
    } else if (BUILD) {
      if (sa > 0.f) {
        float G[NC];
        load_row4<KQ>(S.G, R, G);
#pragma unroll
        for (int j = 0; j < NC; ++j) {
          const int32_t col = 4 * (lane + kWave * (j / 4)) + (j & 3);
          G[j] = col < R ? G[j] : -INFINITY;
        }
        const float fi = row_exact4<NC>(x, G, vc, sa, kappa);
        if (lane == 0) S.F[i] = fi;
        u = 1.f;
      } else {
#pragma unroll
        for (int j = 0; j < NC; ++j) x[j] = 0.f;
        if (lane == 0) S.F[i] = -INFINITY;
      }
      store_row4<KQ>(S.K + (int64_t)i * R, R, x);
    }
    if (step && sa > 0.f) {
      float y = 0.f;
#pragma unroll
      for (int j = 0; j < NC; ++j) y = __builtin_fmaf(x[j], vc[j], y);
      y = lanes_sum(y);
      u = sa * frcp(y);
      if (!linear && !in_range(u)) {  // uniform: every lane holds the same y
        bad |= 1u << k;    // updated after the stream, from C
        u = 0.f;
      }
    }
#pragma unroll
    for (int j = 0; j < NC; ++j) cs[j] = __builtin_fmaf(u, x[j], cs[j]);
    if (lane == k) uo = u;
  };
  Unrolled<kDnWaveRows>::run(row);
  // rows whose u left the range: the exact log-domain update from the row of
  // C (u = 1), added to the column sums after the streamed rows
  for (uint32_t m = (uint32_t)__builtin_amdgcn_readfirstlane((int)bad); m; m &= m - 1) {
    const int k = __builtin_ctz(m);
    const int32_t i = r0 + k;
    const float sa = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sal), k));
    float x[NC], G[NC];
    load_row4<KQ>(Cb + (int64_t)i * R, R, x);
    load_row4<KQ>(S.G, R, G);
#pragma unroll
    for (int j = 0; j < NC; ++j) {
      const int32_t col = 4 * (lane + kWave * (j / 4)) + (j & 3);
      G[j] = col < R ? G[j] : -INFINITY;
    }
    const float fi = row_exact4<NC>(x, G, vc, sa, kappa);
    store_row4<KQ>(S.K + (int64_t)i * R, R, x);
    if (lane == 0) S.F[i] = fi;
#pragma unroll
    for (int j = 0; j < NC; ++j) cs[j] += x[j];
    if (lane == k) uo = 1.f;
  }
  if (lane < nrows) S.u[r0 + lane] = uo;
  store_row4<KQ>(wpart + (int64_t)wid * R, R, cs);
  __syncthreads();
  for (int32_t q = tid; q < R / 4; q += kDnThreads) {
    float4 a = reinterpret_cast<const float4*>(wpart)[q];
#pragma unroll
    for (int w = 1; w < kDnWaves; ++w) {
      const float4 b = reinterpret_cast<const float4*>(wpart + w * R)[q];
      a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
    }
    reinterpret_cast<float4*>(S.part + (int64_t)blk * R)[q] = a;
  }
}

// One column half-step for 16 columns of a problem: the 16 thread groups add
// a sixteenth of the row blocks' partials each (64-byte segments per group)
// and the first 16 threads set v_j from the group sums (added in group
// order).  A column whose v_j leaves [2^-60, 2^60] goes to a list in LDS; the
// four waves then take the listed columns one each for the exact log-domain
// update from C (all RPL loads of a lane in flight at once), with the column
// of K~ rebuilt.  Sixteen columns per block spread these updates over many
// waves when whole batches of columns leave the range together.
template <int RPL>
__global__ void __launch_bounds__(kDnThreads) dense_col_kernel(SkParams p, float kappa) {
  constexpr int G = kDnThreads / kDnColBlock;
  __shared__ float ps[G][kDnColBlock];
  __shared__ int32_t fixl[kDnColBlock];
  __shared__ int32_t nfix;
  const int32_t R = p.R, NB = dense_blocks(R);
  const int32_t chunks = (R + kDnColBlock - 1) / kDnColBlock;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
  const int grp = tid / kDnColBlock, cl = tid % kDnColBlock;
  const int64_t pb = blockIdx.x / chunks;
  const int32_t j = (int32_t)(blockIdx.x % chunks) * kDnColBlock + cl;
  if (p.stream_flag[pb] != 0) return;  // uniform per block
  const DenseState S = dense_state(p, pb);
  const float dj = tid < kDnColBlock && j < R ? p.b[pb * R + j] : 0.f;  // in flight with the partials
  float x = 0.f;
  if (j < R)
    for (int32_t t = NB * grp / G; t < NB * (grp + 1) / G; ++t) x += S.part[(int64_t)t * R + j];
  ps[grp][cl] = x;
  if (tid == 0) nfix = 0;
  __syncthreads();
  if (tid < kDnColBlock && j < R) {
    if (!(dj > 0.f)) {
      // no demand: no flow into this column, and its entries of K~ are zero
      // in every later rebuild (G_j = -inf), so none can overflow
      S.v[j] = 0.f;
      S.G[j] = -INFINITY;
    } else {
      float xs = ps[0][cl];
#pragma unroll
      for (int g = 1; g < G; ++g) xs += ps[g][cl];
      const float vn = dj * frcp(xs);
      if (in_range(vn) || (p.flags & TAOT_SK_LINEAR)) S.v[j] = vn;
      else fixl[atomicAdd(&nfix, 1)] = j;
    }
  }
  __syncthreads();
  const float* Cb = p.C + pb * p.C_stride;
  for (int32_t q = wid; q < nfix; q += kDnWaves) {
    const int32_t c = fixl[q];
    const float dc = p.b[pb * R + c];
    float cc[RPL], fl[RPL], xx[RPL];
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      const int32_t i = lane + kWave * k;
      cc[k] = 0.f;
      fl[k] = -INFINITY;
      float uu = 0.f;
      if (i < R) {
        cc[k] = Cb[(int64_t)i * R + c];
        fl[k] = S.F[i];
        uu = S.u[i];
      }
      xx[k] = uu > 0.f ? (fl[k] + flog2(uu)) - cc[k] * kappa : -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int k = 0; k < RPL; ++k) mx = fmaxf(mx, xx[k]);
    mx = wave_max(mx);
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < RPL; ++k)
      if (xx[k] != -INFINITY) s += fexp2(xx[k] - mx);
    s = wave_sum(s);
    const float gc = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(flog2(dc) - (mx + flog2(s)))));
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      const int32_t i = lane + kWave * k;
      if (i < R) S.K[(int64_t)i * R + c] = fl[k] != -INFINITY ? fexp2((fl[k] + gc) - cc[k] * kappa) : 0.f;
    }
    if (lane == 0) {
      S.G[c] = gc;
      S.v[c] = 1.f;
    }
  }
}

// The plan of the row block, T_ij = u_i K~_ij v_j, and its column sums for
// the column cap.
__global__ void __launch_bounds__(kDnThreads) dense_plan_kernel(SkParams p) {
  const int32_t R = p.R, RB = kDnRowBlock, NB = dense_blocks(R);
  const int64_t pb = blockIdx.x / NB;
  const int32_t blk = blockIdx.x % NB;
  if (p.stream_flag[pb] != 0) return;
  const DenseState S = dense_state(p, pb);
  float* Tb = p.T + pb * R * R;
  const int32_t r0 = blk * RB, r1 = r0 + RB < R ? r0 + RB : R;
  for (int32_t j = threadIdx.x; j < R; j += kDnThreads) {
    const float vj = S.v[j];
    float c = 0.f;
    for (int32_t i = r0; i < r1; ++i) {
      const float t = S.u[i] * S.K[(int64_t)i * R + j] * vj;
      Tb[(int64_t)i * R + j] = t;
      c += t;
    }
    S.part[(int64_t)blk * R + j] = c;
  }
}

// Column-cap factors (into the partials' first row), f, g and the status.
__global__ void __launch_bounds__(kDnThreads) dense_out_kernel(SkParams p, int32_t have_sums) {
  const int32_t R = p.R, NB = dense_blocks(R);
  const int32_t chunks = (R + kDnThreads - 1) / kDnThreads;
  const int64_t pb = blockIdx.x / chunks;
  const int32_t j = (int32_t)(blockIdx.x % chunks) * kDnThreads + threadIdx.x;
  if (p.stream_flag[pb] != 0 || j >= R) return;
  const DenseState S = dense_state(p, pb);
  const float dj = p.b[pb * R + j];
  if (have_sums) {
    float c = 0.f;
    for (int32_t t = 0; t < NB; ++t) c += S.part[(int64_t)t * R + j];
    S.part[j] = fminf(1.f, dj / (c + 1e-12f));
  }
  const float to_nat = p.eps * kLn2;
  const float ui = S.u[j], vj = S.v[j];
  if (p.f) p.f[pb * R + j] = ui > 0.f ? (S.F[j] + flog2(ui)) * to_nat : -INFINITY;
  if (p.g) p.g[pb * R + j] = vj > 0.f ? (S.G[j] + flog2(vj)) * to_nat : -INFINITY;
  if (j == 0 && p.status) p.status[pb] = TAOT_ST_STREAMED;
}

// T_ij *= cap_j over the rows of a row block, the thread's columns held in
// registers (16-byte accesses when R % 4 == 0).
__global__ void __launch_bounds__(kDnThreads) dense_cap_kernel(SkParams p) {
  const int32_t R = p.R, RB = kDnRowBlock, NB = dense_blocks(R);
  const int64_t pb = blockIdx.x / NB;
  const int32_t blk = blockIdx.x % NB;
  if (p.stream_flag[pb] != 0) return;
  const DenseState S = dense_state(p, pb);
  float* Tb = p.T + pb * R * R;
  const int32_t r0 = blk * RB, r1 = r0 + RB < R ? r0 + RB : R;
  if ((R & 3) == 0) {
    for (int32_t q = threadIdx.x; q < R / 4; q += kDnThreads) {
      const float4 cap = reinterpret_cast<const float4*>(S.part)[q];
      for (int32_t i = r0; i < r1; ++i) {
        float4* t = reinterpret_cast<float4*>(Tb + (int64_t)i * R) + q;
        float4 x = *t;
        x.x *= cap.x; x.y *= cap.y; x.z *= cap.z; x.w *= cap.w;
        *t = x;
      }
    }
  } else {
    for (int32_t j = threadIdx.x; j < R; j += kDnThreads) {
      const float cap = S.part[j];
      for (int32_t i = r0; i < r1; ++i) Tb[(int64_t)i * R + j] *= cap;
    }
  }
}

template <bool BUILD>
taot_status launch_rows(const SkParams& p, float kappa, unsigned grid, hipStream_t stream) {
  const int32_t R = p.R;
  if ((R & 3) == 0 && (reinterpret_cast<uintptr_t>(p.C) & 15u) == 0) {
    const size_t lds = (size_t)kDnWaves * R * sizeof(float);
    const int kq = dense_kq(R);
#define TAOT_DN_ROWW(K)                                                                                        \
  if (kq == K) {                                                                                             \
    hipLaunchKernelGGL((dense_roww_kernel<K, BUILD>), dim3(grid), dim3(kDnThreads), lds, stream, p, kappa); \
    return TAOT_OK;                                                                                          \
  }
    TAOT_DN_ROWW(1)
    TAOT_DN_ROWW(2)
    TAOT_DN_ROWW(4)
    TAOT_DN_ROWW(8)
#undef TAOT_DN_ROWW
    return TAOT_ERR_UNSUPPORTED;
  }
  const int kpt = dense_kpt(R);
#define TAOT_DN_ROW(K)                                                                                        \
  if (kpt == K) {                                                                                             \
    hipLaunchKernelGGL((dense_row_kernel<1, K, BUILD>), dim3(grid), dim3(kDnThreads), 0, stream, p, kappa); \
    return TAOT_OK;                                                                                           \
  }
  TAOT_DN_ROW(1)
  TAOT_DN_ROW(2)
  TAOT_DN_ROW(4)
  TAOT_DN_ROW(8)
#undef TAOT_DN_ROW
  return TAOT_ERR_UNSUPPORTED;
}

}  // namespace

size_t dense_state_floats(int32_t R) { return (size_t)5 * R + (size_t)dense_blocks(R) * R; }

taot_status launch_dense(const SkParams& p, hipStream_t stream) {
  const int32_t R = p.R, B = p.B;
  if (R < 1 || R > TAOT_MAX_RANKS) return TAOT_ERR_UNSUPPORTED;
  const float kappa = kLog2e / p.eps;
  hipLaunchKernelGGL(dense_init_kernel, dim3((unsigned)B), dim3(kDnThreads), 0, stream, p);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  const unsigned row_grid = (unsigned)((int64_t)B * dense_blocks(R));
  const unsigned col_grid = (unsigned)((int64_t)B * ((R + kDnColBlock - 1) / kDnColBlock));
  const unsigned out_grid = (unsigned)((int64_t)B * ((R + kDnThreads - 1) / kDnThreads));
  for (int32_t it = 1; it <= p.iters; ++it) {
    const taot_status st = it == 1 ? launch_rows<true>(p, kappa, row_grid, stream)
                                   : launch_rows<false>(p, kappa, row_grid, stream);
    if (st != TAOT_OK) return st;
    if (R <= 16 * kWave)
      hipLaunchKernelGGL(dense_col_kernel<16>, dim3(col_grid), dim3(kDnThreads), 0, stream, p, kappa);
    else
      hipLaunchKernelGGL(dense_col_kernel<32>, dim3(col_grid), dim3(kDnThreads), 0, stream, p, kappa);
  }
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  const bool colcap = p.T && !(p.flags & TAOT_SK_NO_COLCAP);
  if (p.T) {
    hipLaunchKernelGGL(dense_plan_kernel, dim3(row_grid), dim3(kDnThreads), 0, stream, p);
    if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  }
  hipLaunchKernelGGL(dense_out_kernel, dim3(out_grid), dim3(kDnThreads), 0, stream, p, colcap ? 1 : 0);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  if (colcap) {
    hipLaunchKernelGGL(dense_cap_kernel, dim3(row_grid), dim3(kDnThreads), 0, stream, p);
    if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  }
  return TAOT_OK;
}

}  // namespace taot
