// Steps 1-2 of the planner: expert-load histogram and the load marginals.
//
// Sec. 3.1 / A.1 define n_re (tokens rank r sends to expert e), the rank load
// l_r = sum_{e in E_r} sum_r' n_r'e, the mean, excess/spare and rho; Sec. A.3
// defines the spill of each expert by cumulative-excess differencing over the
// experts of a rank sorted by ascending load.  All of it is integer work and
// is exact; rho and alpha are one rounded fp64 division each.
//
// Kernels
//   home_csr_kernel    (1 block)      rank -> experts lists of the home map
//                                     (counts, scan, placement; the order of
//                                     a rank's list is not used).
//   histogram_kernel   (B*R blocks)   one (problem, source rank) row per block;
//                                     streams the ids once (HBM-bound) into LDS
//                                     counters privatised per lane group (32-bit,
//                                     or two 16-bit counters per word when the
//                                     experts are many and a row short enough);
//                                     writes a row's counts as 16-bit pairs when
//                                     the row is short enough.
//   expert_load_kernel (B*E/256)      x_e = sum_r n_re: reads n once, coalesced,
//                                     four experts per lane, rows over the waves;
//                                     widens 16-bit pairs to n in place.
//   marginals_kernel   (B blocks)     loads, mean, excess/spare, rho, alpha,
//                                     spill from x.
#include <mutex>

#include "common.h"

namespace taot {
namespace {

constexpr int kCsrThreads = 1024;
constexpr int kHistThreads = 256;
constexpr int kHistUnroll = 4;
constexpr int kMargThreads = 256;
constexpr int kColThreads = 256;
constexpr int kColExperts = 4 * kWave;         // experts per expert_load_kernel block
constexpr int kHistLdsWords = 16384;           // 64 KiB of 32-bit counters per block when possible
constexpr int kHistLdsWords16 = 8200;          // about 32 KiB of 16-bit counter pairs
constexpr int kHist16MinCopies = 4;            // 16-bit counters when 32-bit ones allow fewer copies

typedef int32_t v4i __attribute__((ext_vector_type(4)));
typedef uint32_t v2u __attribute__((ext_vector_type(2)));

// rank_ptr[R+1], rank_exp[E]: experts of rank r are rank_exp[rank_ptr[r] ..
// rank_ptr[r+1]) in no particular order.  bad_home = 1 if some home is
// outside [0, R).  Also clears the per-problem counts of skipped ids,
// bad_prob[B].
__global__ void __launch_bounds__(kCsrThreads)
home_csr_kernel(const int32_t* __restrict__ home, int32_t B, int32_t R, int32_t E, int32_t* __restrict__ rank_ptr,
                int32_t* __restrict__ rank_exp, int32_t* __restrict__ bad_home,
                unsigned long long* __restrict__ bad_prob) {
  __shared__ int32_t cnt[TAOT_MAX_RANKS];
  __shared__ int32_t wtot[kCsrThreads / kWave];
  __shared__ int32_t bad;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
  if (tid == 0) bad = 0;
  for (int32_t r = tid; r < R; r += kCsrThreads) cnt[r] = 0;
  __syncthreads();
  for (int32_t e = tid; e < E; e += kCsrThreads) {
    const int32_t h = home[e];
    if (h < 0 || h >= R) bad = 1;
    else atomicAdd(&cnt[h], 1);
  }
  __syncthreads();
  // exclusive scan: thread t takes ranks [t*seg, t*seg + seg)
  constexpr int kSeg = (TAOT_MAX_RANKS + kCsrThreads - 1) / kCsrThreads;
  const int32_t lo = tid * kSeg;
  int32_t mine = 0;
#pragma unroll
  for (int k = 0; k < kSeg; ++k) mine += lo + k < R ? cnt[lo + k] : 0;
  int32_t incl = mine;  // inclusive scan over the wave
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int32_t y = __shfl_up(incl, o, kWave);
    incl += lane >= o ? y : 0;
  }
  if (lane == kWave - 1) wtot[wid] = incl;
  __syncthreads();
  int32_t off = incl - mine;
  for (int w = 0; w < wid; ++w) off += wtot[w];
#pragma unroll
  for (int k = 0; k < kSeg; ++k) {
    if (lo + k < R) {
      const int32_t c = cnt[lo + k];
      rank_ptr[lo + k] = off;
      cnt[lo + k] = off;  // now the placement cursor
      off += c;
    }
  }
  if (lo < R && lo + kSeg >= R) rank_ptr[R] = off;  // the thread holding the last rank
  __syncthreads();
  for (int32_t e = tid; e < E; e += kCsrThreads) {
    const int32_t h = home[e];
    if (h >= 0 && h < R) rank_exp[atomicAdd(&cnt[h], 1)] = e;
  }
  if (tid == 0) bad_home[0] = bad;
  for (int32_t b = tid; b < B; b += kCsrThreads) bad_prob[b] = 0;
}

// One block per (problem, source rank) row of N ids.  LDS holds `copies`
// private histograms; lane group (tid & (copies-1)) owns one copy, which
// spreads the heavy Zipf bins over distinct LDS addresses.  Bin E of a copy
// is where ids outside [0, E) are counted, so the count carries no branch.
// With PACK16 two experts share a 32-bit word (expert e in half e & 1 of
// word e >> 1); the host takes this form only when no copy can count past
// 65535 in one half (a row short enough for the number of copies), and it
// doubles the copies that fit the LDS.  Otherwise a copy is E+1 words; the
// extra word also rotates banks between copies.
//
// Ids are read exactly once, so they stream past the caches.  The bulk of a
// row goes in batches of kHistUnroll 16-byte loads per thread, none of them
// predicated, with the next batch in flight while the current one is counted
// (two register sets, a and b, take turns).  The first batch is issued before
// the counters are cleared.
template <bool PACK16>
__global__ void __launch_bounds__(kHistThreads)
histogram_kernel(const int32_t* __restrict__ ids, int64_t N, int32_t R, int32_t E, int32_t copies, bool half,
                 int32_t* __restrict__ n, unsigned long long* __restrict__ bad_prob) {
  extern __shared__ int32_t bins[];
  const int64_t row = blockIdx.x;
  const int32_t stride = PACK16 ? (E >> 1) + 1 : E + 1;
  const int32_t words = copies * stride;
  int32_t* my = bins + (int32_t)(threadIdx.x & (copies - 1)) * stride;
  const int32_t* src = ids + row * N;
  const uint32_t uE = (uint32_t)E;
  auto count = [&](int32_t q) {
    const int32_t e = (uint32_t)q < uE ? q : E;
    if constexpr (PACK16) atomicAdd(&my[e >> 1], (e & 1) ? 0x10000 : 1);
    else atomicAdd(&my[e], 1);
  };
  auto count4 = [&](const v4i& v) {
    count(v.x);
    count(v.y);
    count(v.z);
    count(v.w);
  };
  const bool vec = (N % 4 == 0) && ((reinterpret_cast<uintptr_t>(src) & 15u) == 0);
  const v4i* s4 = reinterpret_cast<const v4i*>(src);
  constexpr int64_t kStep = (int64_t)kHistThreads * kHistUnroll;
  const int64_t nb = vec ? (N / 4) / kStep : 0;  // full batches
  const v4i* p = s4 + threadIdx.x;
  v4i a[kHistUnroll], b[kHistUnroll];
  if (nb > 0) {
#pragma unroll
    for (int u = 0; u < kHistUnroll; ++u) a[u] = __builtin_nontemporal_load(p + u * kHistThreads);
  }
  for (int32_t i = threadIdx.x; i < words; i += kHistThreads) bins[i] = 0;
  __syncthreads();
  if (nb > 0) {
    int64_t m = 0;  // batch held in a (even turns) or b (odd turns)
    for (;;) {
      if (m + 1 == nb) {
#pragma unroll
        for (int u = 0; u < kHistUnroll; ++u) count4(a[u]);
        break;
      }
      p += kStep;
#pragma unroll
      for (int u = 0; u < kHistUnroll; ++u) b[u] = __builtin_nontemporal_load(p + u * kHistThreads);
#pragma unroll
      for (int u = 0; u < kHistUnroll; ++u) count4(a[u]);
      if (++m + 1 == nb) {
#pragma unroll
        for (int u = 0; u < kHistUnroll; ++u) count4(b[u]);
        break;
      }
      p += kStep;
#pragma unroll
      for (int u = 0; u < kHistUnroll; ++u) a[u] = __builtin_nontemporal_load(p + u * kHistThreads);
#pragma unroll
      for (int u = 0; u < kHistUnroll; ++u) count4(b[u]);
      ++m;
    }
  }
  // what the full batches left: the vector tail, or the whole row when it is
  // not 16-byte aligned
  if (vec) {
    for (int64_t i = nb * kStep + threadIdx.x; i < N / 4; i += kHistThreads)
      count4(__builtin_nontemporal_load(&s4[i]));
  } else {
    for (int64_t i = threadIdx.x; i < N; i += kHistThreads) count(src[i]);
  }
  __syncthreads();
  // The counts are not read again by this kernel, and ordinary stores of them
  // interleaved with the id stream cost far more read bandwidth than their
  // size: they are written past the caches too, and with `half` in half the
  // bytes (the layout below, which expert_load_kernel<true> widens in place).
  // Skipped ids are rare, so their count reaches memory only when it is not
  // zero.
  auto total = [&](int32_t e) {
    int32_t s = 0;
    if constexpr (PACK16) {
      const int sh = (e & 1) * 16;
      for (int32_t c = 0; c < copies; ++c) s += (int32_t)(((uint32_t)bins[c * stride + (e >> 1)] >> sh) & 0xFFFFu);
    } else {
      for (int32_t c = 0; c < copies; ++c) s += bins[c * stride + e];
    }
    return s;
  };
  int32_t* dst = n + row * E;
  if (half) {
    // Experts 2q and 2q+1 share a word; pair q is pair j = q mod 128 of the
    // kColExperts-wide chunk c = q / 128, at word j of the chunk's part of
    // the row.  A count above 65534 is stored as 0xFFFF, its value at word
    // w-1-j of the chunk (w experts wide), in the half the pairs leave free.
    // The host takes this form only for rows of fewer than 2 * 65535 ids, so
    // a row has at most one such count and the two halves of a pair never
    // both need the spare word.
    for (int32_t q = threadIdx.x; 2 * q < E; q += kHistThreads) {
      const int32_t c = q >> 7, j = q & 127;
      int32_t* chunk = dst + c * kColExperts;
      const int32_t lo = total(2 * q), hi = total(2 * q + 1);
      const uint32_t word = (uint32_t)min(lo, 0xFFFF) | ((uint32_t)min(hi, 0xFFFF) << 16);
      __builtin_nontemporal_store((int32_t)word, &chunk[j]);
      if (max(lo, hi) >= 0xFFFF) chunk[min(kColExperts, E - c * kColExperts) - 1 - j] = max(lo, hi);
    }
    if (threadIdx.x == 0) {
      const int32_t s = total(E);
      if (s != 0) atomicAdd(&bad_prob[row / R], (unsigned long long)s);
    }
    return;
  }
  for (int32_t e = threadIdx.x; e <= E; e += kHistThreads) {
    const int32_t s = total(e);
    if (e < E)
      __builtin_nontemporal_store(s, &dst[e]);
    else if (s != 0)
      atomicAdd(&bad_prob[row / R], (unsigned long long)s);
  }
}

// x_e = sum_r n_re for a block of kColExperts experts of one problem: lane l
// of every wave sums experts 4l .. 4l+3 of the block (one 16-byte load per
// row when rows are 16-byte aligned, else four 4-byte loads), wave w rows
// w, w + 4, ...; the waves' partial sums meet in LDS.  Integer sums: exact in
// any order.
//
// HALF: the histogram left the block's counts of each row as 16-bit pairs
// (see histogram_kernel); lane l reads the pair words 2l and 2l+1 (8 bytes),
// takes a count stored as 0xFFFF from its spare word, and writes the four
// counts back as 32-bit words 4l .. 4l+3.  One wave reads and rewrites the
// whole block of a row, and its stores use the values of all its loads, so
// every word of the row is read before any is overwritten; other waves and
// blocks touch other rows or other blocks.
template <bool HALF>
__global__ void __launch_bounds__(kColThreads)
expert_load_kernel(int32_t* __restrict__ n, int32_t R, int32_t E, int64_t* __restrict__ load_e) {
  constexpr int kWaves = kColThreads / kWave;
  constexpr int kRowsInFlight = 8;
  __shared__ long long part[kWaves][kColExperts];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
  const int32_t chunks = (E + kColExperts - 1) / kColExperts;
  const int64_t b = blockIdx.x / chunks;
  const int32_t e0 = (int32_t)(blockIdx.x % chunks) * kColExperts + 4 * lane;
  int32_t* nb = n + b * (int64_t)R * E;
  const bool vec = (E % 4 == 0) && ((reinterpret_cast<uintptr_t>(n) & 15u) == 0);
  int64_t s[4] = {0, 0, 0, 0};
  if (e0 < E) {
    auto add_row = [&](int32_t r) {
      if constexpr (HALF) {
        int32_t* blk = nb + (int64_t)r * E + (e0 - 4 * lane);
        const int32_t w = min(kColExperts, E - (e0 - 4 * lane));
        const v2u p = *reinterpret_cast<const v2u*>(blk + 2 * lane);
        int32_t c[4] = {(int32_t)(p.x & 0xFFFFu), (int32_t)(p.x >> 16), (int32_t)(p.y & 0xFFFFu),
                        (int32_t)(p.y >> 16)};
        if (c[0] == 0xFFFF || c[1] == 0xFFFF) {
          const int32_t big = blk[w - 1 - 2 * lane];
          c[0] = c[0] == 0xFFFF ? big : c[0];
          c[1] = c[1] == 0xFFFF ? big : c[1];
        }
        if (c[2] == 0xFFFF || c[3] == 0xFFFF) {
          const int32_t big = blk[w - 2 - 2 * lane];
          c[2] = c[2] == 0xFFFF ? big : c[2];
          c[3] = c[3] == 0xFFFF ? big : c[3];
        }
        *reinterpret_cast<v4i*>(blk + 4 * lane) = v4i{c[0], c[1], c[2], c[3]};
        s[0] += c[0]; s[1] += c[1]; s[2] += c[2]; s[3] += c[3];
        return;
      }
      const int32_t* q = nb + (int64_t)r * E + e0;
      if (vec) {
        const v4i v = *reinterpret_cast<const v4i*>(q);
        s[0] += v.x; s[1] += v.y; s[2] += v.z; s[3] += v.w;
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) s[k] += e0 + k < E ? q[k] : 0;
      }
    };
    int32_t r = wid;
    for (; r + (kRowsInFlight - 1) * kWaves < R; r += kRowsInFlight * kWaves) {
#pragma unroll
      for (int u = 0; u < kRowsInFlight; ++u) add_row(r + u * kWaves);
    }
    for (; r < R; r += kWaves) add_row(r);
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) part[wid][4 * lane + k] = s[k];
  __syncthreads();
  const int32_t e = (int32_t)(blockIdx.x % chunks) * kColExperts + tid;
  if (tid < kColExperts && e < E) {
    int64_t t = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) t += part[w][tid];
    load_e[b * E + e] = t;
  }
}

// Optional hot/cold rank lists of the marginals: [B][R] ascending lists
// (padded with -1) and [B] counts, each nullable.
struct HotCold {
  int32_t* hot_idx;
  int32_t* cold_idx;
  int32_t* hot_cnt;
  int32_t* cold_cnt;
};

// Exclusive positions of two flags among the kMargThreads threads (ascending
// thread id) and their totals.  All threads must call it.
__device__ __forceinline__ void block_scan2(bool f0, bool f1, int32_t (*cnt)[kMargThreads / kWave], int32_t& p0,
                                            int32_t& p1, int32_t& t0, int32_t& t1) {
  const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
  const uint64_t m0 = __ballot(f0), m1 = __ballot(f1);
  const uint64_t below = (1ull << lane) - 1ull;
  if (lane == 0) {
    cnt[0][wid] = __popcll(m0);
    cnt[1][wid] = __popcll(m1);
  }
  __syncthreads();
  int32_t o0 = 0, o1 = 0, s0 = 0, s1 = 0;
  for (int w = 0; w < kMargThreads / kWave; ++w) {
    const int32_t a = cnt[0][w], c = cnt[1][w];
    o0 += w < wid ? a : 0;
    o1 += w < wid ? c : 0;
    s0 += a;
    s1 += c;
  }
  __syncthreads();  // every thread has read cnt before the next call rewrites it
  p0 = o0 + __popcll(m0 & below);
  p1 = o1 + __popcll(m1 & below);
  t0 = s0;
  t1 = s1;
}

// One block per problem; x_e comes from expert_load_kernel.
__global__ void __launch_bounds__(kMargThreads)
marginals_kernel(int32_t R, int32_t E, const int32_t* __restrict__ home, const int32_t* __restrict__ rank_ptr,
                 const int32_t* __restrict__ rank_exp, const int32_t* __restrict__ bad_home,
                 const unsigned long long* __restrict__ bad_prob, int64_t* __restrict__ load_e,
                 int64_t* __restrict__ load_r, int64_t* __restrict__ excess, int64_t* __restrict__ spare,
                 int64_t* __restrict__ spill, float* __restrict__ supply, float* __restrict__ demand,
                 double* __restrict__ rho, double* __restrict__ alpha, int64_t* __restrict__ bad_ids,
                 HotCold hc, uint32_t* __restrict__ status) {
  const int64_t b = blockIdx.x;
  const int tid = threadIdx.x;
  __shared__ int64_t red_s[kMargThreads / kWave], red_m[kMargThreads / kWave];
  __shared__ int32_t scan_cnt[2][kMargThreads / kWave];
  __shared__ int64_t sh_L, sh_max;
  const bool home_bad = bad_home[0] != 0;
  const int64_t skipped = (int64_t)bad_prob[b];  // ids of this problem outside [0, E)

  int64_t* xe = load_e + b * E;
  if (home_bad) {
    for (int32_t e = tid; e < E; e += kMargThreads) { xe[e] = 0; spill[b * E + e] = 0; }
    for (int32_t r = tid; r < R; r += kMargThreads) {
      load_r[b * R + r] = 0; excess[b * R + r] = 0; spare[b * R + r] = 0;
      if (supply) supply[b * R + r] = 0.f;
      if (demand) demand[b * R + r] = 0.f;
    }
    for (int32_t r = tid; r < R; r += kMargThreads) {
      if (hc.hot_idx) hc.hot_idx[b * R + r] = -1;
      if (hc.cold_idx) hc.cold_idx[b * R + r] = -1;
    }
    if (tid == 0) {
      if (rho) rho[b] = 0.0;
      alpha[b] = 0.0;
      if (bad_ids) bad_ids[b] = skipped;
      if (hc.hot_cnt) hc.hot_cnt[b] = 0;
      if (hc.cold_cnt) hc.cold_cnt[b] = 0;
      if (status) status[b] = TAOT_ST_BAD_INPUT | (skipped ? TAOT_ST_BAD_ID : 0u);
    }
    return;
  }

  // rank loads, total and maximum
  int64_t ls = 0, lm = 0;
  for (int32_t r = tid; r < R; r += kMargThreads) {
    int64_t s = 0;
    for (int32_t q = rank_ptr[r]; q < rank_ptr[r + 1]; ++q) s += xe[rank_exp[q]];
    load_r[b * R + r] = s;
    ls += s;
    lm = s > lm ? s : lm;
  }
  ls = wave_sum_i64(ls);
  lm = wave_max_i64(lm);
  if ((tid & (kWave - 1)) == 0) { red_s[tid / kWave] = ls; red_m[tid / kWave] = lm; }
  __syncthreads();
  if (tid == 0) {
    int64_t s = 0, m = 0;
    for (int i = 0; i < kMargThreads / kWave; ++i) { s += red_s[i]; m = red_m[i] > m ? red_m[i] : m; }
    sh_L = s;
    sh_max = m;
  }
  __syncthreads();
  const int64_t L = sh_L;
  const int64_t mean = L / R;  // integer mean floor(L / R)
  for (int32_t r = tid; r < R; r += kMargThreads) {
    const int64_t l = load_r[b * R + r];
    const int64_t ex = l > mean ? l - mean : 0;
    const int64_t sp = mean > l ? mean - l : 0;
    excess[b * R + r] = ex;
    spare[b * R + r] = sp;
    if (supply) supply[b * R + r] = (float)ex;
    if (demand) demand[b * R + r] = (float)sp;
  }
  // the hot and cold sets H = {r : l_r > m}, C = {r : l_r < m} (Sec. A.1) as
  // ascending rank lists padded with -1 (each thread reads back the loads it
  // wrote above: same rank stride)
  if (hc.hot_idx || hc.cold_idx || hc.hot_cnt || hc.cold_cnt) {
    int32_t nh = 0, nc = 0;
    for (int32_t base = 0; base < R; base += kMargThreads) {
      const int32_t r = base + tid;
      const int64_t l = r < R ? load_r[b * R + r] : mean;
      int32_t ph, pc, th, tc;
      block_scan2(l > mean, l < mean, scan_cnt, ph, pc, th, tc);
      if (l > mean && hc.hot_idx) hc.hot_idx[b * R + nh + ph] = r;
      if (l < mean && hc.cold_idx) hc.cold_idx[b * R + nc + pc] = r;
      nh += th;
      nc += tc;
    }
    for (int32_t r = tid; r < R; r += kMargThreads) {
      if (hc.hot_idx && r >= nh) hc.hot_idx[b * R + r] = -1;
      if (hc.cold_idx && r >= nc) hc.cold_idx[b * R + r] = -1;
    }
    if (tid == 0) {
      if (hc.hot_cnt) hc.hot_cnt[b] = nh;
      if (hc.cold_cnt) hc.cold_cnt[b] = nc;
    }
  }
  if (tid == 0) {
    if (rho) rho[b] = L > 0 ? (double)((int64_t)R * sh_max - L) / (double)L : 0.0;
    alpha[b] = (double)L / (double)E;
    if (bad_ids) bad_ids[b] = skipped;
    if (status) status[b] = skipped ? TAOT_ST_BAD_ID : 0u;
  }
  // spill: prefix of the expert's rank in ascending (x, id) order, then
  // sigma_k - sigma_{k-1} with sigma = max(prefix - mean, 0)
  for (int32_t e = tid; e < E; e += kMargThreads) {
    const int32_t h = home[e];
    const int64_t x = xe[e];
    int64_t P = 0;
    for (int32_t q = rank_ptr[h]; q < rank_ptr[h + 1]; ++q) {
      const int32_t e2 = rank_exp[q];
      const int64_t x2 = xe[e2];
      if (x2 < x || (x2 == x && e2 <= e)) P += x2;
    }
    const int64_t hi = P > mean ? P - mean : 0;
    const int64_t lo = P - x > mean ? P - x - mean : 0;
    spill[b * E + e] = hi - lo;
  }
}

struct LoadsWs {
  int32_t* rank_ptr;
  int32_t* rank_exp;
  int32_t* bad_home;
  unsigned long long* bad_prob;
  size_t bytes;
};

LoadsWs carve(void* ws, int32_t B, int32_t R, int32_t E) {
  Carver c{static_cast<char*>(ws)};
  LoadsWs w;
  w.rank_ptr = c.take<int32_t>((size_t)R + 1);
  w.rank_exp = c.take<int32_t>((size_t)E);
  w.bad_home = c.take<int32_t>(1);
  w.bad_prob = c.take<unsigned long long>((size_t)B);
  w.bytes = c.off;
  return w;
}

// Fixed scratch of the allocation-free entry point: the same workspace
// layout as above, in a file-scope device array (one copy per GPU, held until
// the process ends).  Host code never uses the array's name as an address:
// its device address is looked up once per device with hipGetSymbolAddress.
constexpr size_t kScratchBytes = (size_t)1 << 20;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void* scratch_ptr[kMaxDevices] = {};

}  // namespace

size_t plan_loads_ws(int32_t B, int32_t R, int32_t E) { return carve(nullptr, B, R, E).bytes; }

size_t plan_loads_scratch_limit() { return kScratchBytes; }

// Device address of this device's scratch array (looked up on the first call
// per device), or nullptr if the runtime cannot give it.
void* plan_loads_scratch() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    scratch_ptr[dev] = ptr;
  }
  return scratch_ptr[dev];
}

taot_status launch_plan_loads(const int32_t* ids, int32_t B, int32_t R, int64_t N, int32_t E,
                              const int32_t* home, int32_t* n, int64_t* load_e, int64_t* load_r,
                              int64_t* excess, int64_t* spare, int64_t* spill, float* supply,
                              float* demand, double* rho, double* alpha, int64_t* bad_ids,
                              int32_t* hot_idx, int32_t* cold_idx, int32_t* hot_cnt, int32_t* cold_cnt,
                              uint32_t* status, void* ws, hipStream_t stream) {
  if (B == 0) return TAOT_OK;
  LoadsWs w = carve(ws, B, R, E);
  hipLaunchKernelGGL(home_csr_kernel, dim3(1), dim3(kCsrThreads), 0, stream, home, B, R, E, w.rank_ptr,
                     w.rank_exp, w.bad_home, w.bad_prob);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  // counter layout: 32-bit copies of E+1 words while 16 fit the LDS cap;
  // else 16-bit pairs, twice as many copies in half the words, when no copy
  // can count past 65535 (a copy's lane group reads at most N / copies ids
  // plus one 16-byte batch tail per thread)
  int32_t copies = 16;
  while (copies > 1 && (int64_t)copies * (E + 1) > kHistLdsWords) copies >>= 1;
  int32_t copies16 = 16;
  const int64_t stride16 = (E >> 1) + 1;
  while (copies16 > 1 && (int64_t)copies16 * stride16 > kHistLdsWords16) copies16 >>= 1;
  const bool pack16 = copies < kHist16MinCopies && copies16 > copies &&
                      N / copies16 + 4 * kHistUnroll * (kHistThreads / copies16) * 4 <= 65535;
  if (pack16) copies = copies16;
  const size_t lds = (size_t)copies * (pack16 ? stride16 : (E + 1)) * sizeof(int32_t);
  const void* hist = pack16 ? (const void*)histogram_kernel<true> : (const void*)histogram_kernel<false>;
  if (lds > 65536 &&
      hipFuncSetAttribute(hist, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return TAOT_ERR_LAUNCH;
  // counts stored as 16-bit pairs (half the bytes next to the id stream) when
  // the rows are 16-byte aligned and shorter than 2 * 65535 ids
  const bool half = E % 4 == 0 && (reinterpret_cast<uintptr_t>(n) & 15u) == 0 && N < 2 * 65535;
  if (pack16)
    hipLaunchKernelGGL(histogram_kernel<true>, dim3((unsigned)((int64_t)B * R)), dim3(kHistThreads), lds, stream,
                       ids, N, R, E, copies, half, n, w.bad_prob);
  else
    hipLaunchKernelGGL(histogram_kernel<false>, dim3((unsigned)((int64_t)B * R)), dim3(kHistThreads), lds, stream,
                       ids, N, R, E, copies, half, n, w.bad_prob);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  const dim3 col_grid((unsigned)((int64_t)B * ((E + kColExperts - 1) / kColExperts)));
  if (half)
    hipLaunchKernelGGL(expert_load_kernel<true>, col_grid, dim3(kColThreads), 0, stream, n, R, E, load_e);
  else
    hipLaunchKernelGGL(expert_load_kernel<false>, col_grid, dim3(kColThreads), 0, stream, n, R, E, load_e);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  hipLaunchKernelGGL(marginals_kernel, dim3((unsigned)B), dim3(kMargThreads), 0, stream, R, E, home, w.rank_ptr,
                     w.rank_exp, w.bad_home, w.bad_prob, load_e, load_r, excess, spare, spill, supply, demand,
                     rho, alpha, bad_ids, HotCold{hot_idx, cold_idx, hot_cnt, cold_cnt}, status);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  return TAOT_OK;
}

}  // namespace taot
