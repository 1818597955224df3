// Steps 4-5 of the planner: integer replica matching and token split.
//
// Phase 2 (Alg. 2, Sec. A.3): K rounds of column-priority matching.  In each
// inner iteration every unmatched cold rank proposes its best expert under
// the three-level score min(spill, spare) + alpha*B + 0.1*alpha*T_norm, each
// proposed expert keeps its best proposer, and winners take
// g = min(spill, spare) into their slot for this round.
// Phase 3 (Alg. 3, Sec. A.4): Lagrangian auction.  Each round every open slot
// bids for the source rank with the highest bonus minus price among ranks
// still holding tokens of its expert; each rank serves its best bidder with
// min(tokens held, tokens still planned) and raises its price.
//
// Exactness.  All state is integer; scores are fp64 evaluated in the order
// stated in taot.h and compiled without FP contraction; every argmax is
// masked and breaks ties to the lowest index.  Two shortcuts are exact:
//   - a phase stops at the first iteration/round with no proposal/bid, which
//     leaves the state unchanged and so equals running the remaining ones;
//   - a Phase-3 slot re-bids only when the rank it bid for served (its price
//     rose, its stock fell) or ran out of the slot's expert: every other
//     rank's score can only fall and its validity only end, so the previous
//     argmax (including its tie-break) stands.
//
// One workgroup per problem, grid-stride over problems; per-workgroup state
// lives in a slab of the workspace (L2-resident), per-rank auction
// arbitration in LDS.
#include <limits.h>

#include "common.h"

namespace taot {
namespace {

constexpr int kSchThreads = 256;
constexpr int kSchWaves = kSchThreads / kWave;
constexpr int kSchMaxGrid = 1024;

struct SchParams {
  const int32_t* n;
  const int64_t* spill;
  const int64_t* spare;
  const int64_t* excess;
  const double* alpha;
  const int32_t* home;
  const float* T;
  const double* Bpref;
  const double* Bauct;
  int32_t B, R, E, K;
  double price_step;
  int64_t t_max;
  int32_t* slot_expert;
  int64_t* slot_amount;
  int32_t* X;
  int64_t* unfilled;
  int32_t* rounds_used;
  uint32_t* status;
  char* slab;
  int64_t slab_bytes;
  const int32_t* fallback;  // [B] 1 = the one-wave kernel left this problem to us (nullable)
};

struct Slab {
  // Phase 2
  int32_t* cr;        // [R] cold ranks, ascending
  int64_t* spare_p;   // [R]
  int32_t* matched;   // [R]
  int32_t* prop_e;    // [R] proposed candidate index or -1
  double* prop_s;     // [R]
  int32_t* assigned;  // [R*K] candidate index assigned to cold rank rc in round k
  int32_t* ce;        // [E] candidate experts (spill > 0), ascending
  int64_t* spill_p;   // [E]
  int32_t* win;       // [E] winning cold-rank index or -1
  // Phase 3
  int32_t* dmap;      // [E] expert -> distinct slot-expert index or -1
  int32_t* dexp;      // [D] distinct slot experts, ascending
  int32_t* bid;       // [S]
  double* bid_s;      // [S]
  int64_t* Ap;        // [S] tokens still planned
  int32_t* dsl;       // [S] distinct index of the slot's expert or -1
  int32_t* need;      // [S] 1 = recompute the bid
  int32_t* work;      // [S] compacted list of slots to recompute
  int32_t* nprime;    // [D*R] tokens of distinct expert d still held by rank r
  size_t bytes;
};

__host__ __device__ Slab carve_slab(char* base, int32_t R, int32_t E, int32_t K) {
  Carver c{base};
  const int64_t S = (int64_t)R * K;
  const int64_t D = S < E ? S : E;
  Slab s;
  s.cr = c.take<int32_t>(R);
  s.spare_p = c.take<int64_t>(R);
  s.matched = c.take<int32_t>(R);
  s.prop_e = c.take<int32_t>(R);
  s.prop_s = c.take<double>(R);
  s.assigned = c.take<int32_t>((size_t)R * (K > 0 ? K : 1));
  s.ce = c.take<int32_t>(E);
  s.spill_p = c.take<int64_t>(E);
  s.win = c.take<int32_t>(E);
  s.dmap = c.take<int32_t>(E);
  s.dexp = c.take<int32_t>((size_t)(D > 0 ? D : 1));
  s.bid = c.take<int32_t>((size_t)(S > 0 ? S : 1));
  s.bid_s = c.take<double>((size_t)(S > 0 ? S : 1));
  s.Ap = c.take<int64_t>((size_t)(S > 0 ? S : 1));
  s.dsl = c.take<int32_t>((size_t)(S > 0 ? S : 1));
  s.need = c.take<int32_t>((size_t)(S > 0 ? S : 1));
  s.work = c.take<int32_t>((size_t)(S > 0 ? S : 1));
  s.nprime = c.take<int32_t>((size_t)(D > 0 ? D : 1) * R);
  s.bytes = c.off;
  return s;
}

// Exclusive position of `flag` among the kSchThreads threads (ascending
// thread id) and the chunk total.  All threads must call it.
__device__ __forceinline__ int32_t compact_pos(bool flag, int32_t* wave_cnt, int32_t& total) {
  const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
  const uint64_t m = __ballot(flag);
  const int32_t lp = __popcll(m & ((1ull << lane) - 1ull));
  if (lane == 0) wave_cnt[wid] = __popcll(m);
  __syncthreads();
  int32_t off = 0, tot = 0;
  for (int w = 0; w < kSchWaves; ++w) {
    const int32_t c = wave_cnt[w];
    off += w < wid ? c : 0;
    tot += c;
  }
  __syncthreads();
  total = tot;
  return off + lp;
}

// Block-wide OR of a flag.  All threads must call it.
__device__ __forceinline__ bool block_any(bool flag, int32_t* wave_cnt) {
  const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
  const uint64_t m = __ballot(flag);
  if (lane == 0) wave_cnt[wid] = m != 0;
  __syncthreads();
  bool any = false;
  for (int w = 0; w < kSchWaves; ++w) any |= wave_cnt[w] != 0;
  __syncthreads();
  return any;
}

__device__ __forceinline__ uint64_t auction_key(double x) {
  return ordered_key(x == 0.0 ? 0.0 : x);  // -0 and +0 compare equal
}

__global__ void __launch_bounds__(kSchThreads) schedule_kernel(SchParams p) {
  extern __shared__ char lds_raw[];
  __shared__ int32_t wave_cnt[kSchWaves];
  __shared__ int32_t sh_flag;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
  const int32_t R = p.R, E = p.E, K = p.K;
  const int64_t S = (int64_t)R * K;
  // per-rank auction state in LDS
  double* price = reinterpret_cast<double*>(lds_raw);
  uint64_t* rkey = reinterpret_cast<uint64_t*>(price + R);
  int32_t* rwin = reinterpret_cast<int32_t*>(rkey + R);
  int32_t* served = rwin + R;

  Slab sl = carve_slab(p.slab + (int64_t)blockIdx.x * p.slab_bytes, R, E, K);

  for (int64_t b = blockIdx.x; b < p.B; b += gridDim.x) {
    if (p.fallback && p.fallback[b] == 0) continue;  // uniform per block
    const int64_t* spill = p.spill + b * E;
    const int64_t* spare = p.spare + b * R;
    const int64_t* excess = p.excess + b * R;
    const float* Tb = p.T + b * (int64_t)R * R;
    int32_t* se = p.slot_expert + b * S;
    int64_t* sa = p.slot_amount + b * S;
    int32_t* Xb = p.X + b * (int64_t)R * S;
    const double alpha = p.alpha[b];
    const double a2 = 0.1 * alpha;  // weight of the OT hint

    // ---- validation and setup -----------------------------------------------
    if (tid == 0) sh_flag = 0;
    __syncthreads();
    for (int32_t e = tid; e < E; e += kSchThreads) {
      const int32_t h = p.home[e];
      if (h < 0 || h >= R) sh_flag = 1;
    }
    for (int64_t s = tid; s < S; s += kSchThreads) { se[s] = -1; sa[s] = 0; }
    for (int64_t q = tid; q < (int64_t)R * S; q += kSchThreads) Xb[q] = 0;
    __syncthreads();
    if (sh_flag) {
      if (tid == 0) {
        p.unfilled[b] = 0;
        if (p.rounds_used) { p.rounds_used[2 * b] = 0; p.rounds_used[2 * b + 1] = 0; }
        if (p.status) p.status[b] = TAOT_ST_BAD_INPUT;
      }
      __syncthreads();
      continue;
    }

    // candidate experts (spill > 0) and cold ranks (spare > 0), ascending
    int32_t ne = 0, nc = 0;
    for (int32_t base = 0; base < E; base += kSchThreads) {
      const int32_t e = base + tid;
      const bool f = e < E && spill[e] > 0;
      int32_t tot;
      const int32_t pos = compact_pos(f, wave_cnt, tot);
      if (f) { sl.ce[ne + pos] = e; sl.spill_p[ne + pos] = spill[e]; }
      ne += tot;
    }
    for (int32_t base = 0; base < R; base += kSchThreads) {
      const int32_t r = base + tid;
      const bool f = r < R && spare[r] > 0;
      int32_t tot;
      const int32_t pos = compact_pos(f, wave_cnt, tot);
      if (f) { sl.cr[nc + pos] = r; sl.spare_p[nc + pos] = spare[r]; }
      nc += tot;
    }
    for (int64_t q = tid; q < (int64_t)nc * K; q += kSchThreads) sl.assigned[q] = -1;
    __syncthreads();

    // ---- Phase 2: column-priority iterative matching --------------------------
    int32_t used2 = 0;
    for (int32_t k = 0; k < K; ++k) {
      for (int32_t rc = tid; rc < nc; rc += kSchThreads) sl.matched[rc] = 0;
      __syncthreads();
      for (int32_t inner = 0; inner < nc; ++inner) {
        // Step 1: each unmatched cold rank proposes its best candidate expert
        bool proposed = false;
        for (int32_t rc = tid; rc < nc; rc += kSchThreads) {
          int32_t best = -1;
          double bs = -INFINITY;
          const int64_t sp = sl.spare_p[rc];
          if (!sl.matched[rc] && sp > 0) {
            const int32_t r = sl.cr[rc];
            for (int32_t ec = 0; ec < ne; ++ec) {
              const int64_t spl = sl.spill_p[ec];
              if (spl <= 0) continue;
              const int32_t e = sl.ce[ec];
              const int32_t h = p.home[e];
              if (h == r) continue;
              bool taken = false;
              for (int32_t kk = 0; kk < k; ++kk) taken |= sl.assigned[(int64_t)rc * K + kk] == ec;
              if (taken) continue;
              const double q = (double)(spl < sp ? spl : sp);
              const double t1 = alpha * p.Bpref[(int64_t)h * R + r];
              const double ex = (double)excess[h];
              const double tn = (double)Tb[(int64_t)h * R + r] / (ex > kEps0 ? ex : kEps0);
              const double t2 = a2 * tn;
              const double score = (q + t1) + t2;
              if (score > bs) { bs = score; best = ec; }
            }
          }
          sl.prop_e[rc] = best;
          sl.prop_s[rc] = bs;
          proposed |= best >= 0;
        }
        if (!block_any(proposed, wave_cnt)) break;  // nothing can change any more
        // Steps 2-3: each proposed expert keeps its best proposer (lowest rank on ties)
        for (int32_t ec = tid; ec < ne; ec += kSchThreads) {
          int32_t w = -1;
          double ws = -INFINITY;
          for (int32_t rc = 0; rc < nc; ++rc)
            if (sl.prop_e[rc] == ec && sl.prop_s[rc] > ws) { ws = sl.prop_s[rc]; w = rc; }
          sl.win[ec] = w;
        }
        __syncthreads();
        // Step 4: winners take g = min(spill, spare) into slot k of their rank
        for (int32_t ec = tid; ec < ne; ec += kSchThreads) {
          const int32_t w = sl.win[ec];
          if (w < 0) continue;
          const int64_t g = sl.spill_p[ec] < sl.spare_p[w] ? sl.spill_p[ec] : sl.spare_p[w];
          sl.spill_p[ec] -= g;
          sl.spare_p[w] -= g;
          sl.matched[w] = 1;
          sl.assigned[(int64_t)w * K + k] = ec;
          const int64_t s = (int64_t)sl.cr[w] * K + k;
          se[s] = sl.ce[ec];
          sa[s] += g;
        }
        __syncthreads();
        ++used2;
      }
    }

    // ---- Phase 3: Lagrangian auction --------------------------------------------
    for (int32_t e = tid; e < E; e += kSchThreads) sl.dmap[e] = 0;
    __syncthreads();
    for (int64_t s = tid; s < S; s += kSchThreads)
      if (se[s] >= 0) sl.dmap[se[s]] = 1;
    __syncthreads();
    int32_t D = 0;
    for (int32_t base = 0; base < E; base += kSchThreads) {
      const int32_t e = base + tid;
      const bool f = e < E && sl.dmap[e] == 1;
      int32_t tot;
      const int32_t pos = compact_pos(f, wave_cnt, tot);
      if (e < E) sl.dmap[e] = f ? D + pos : -1;
      if (f) sl.dexp[D + pos] = e;
      D += tot;
    }
    __syncthreads();
    const int32_t* nb = p.n + b * (int64_t)R * E;
    for (int64_t q = tid; q < (int64_t)D * R; q += kSchThreads) {
      const int32_t d = (int32_t)(q / R), r = (int32_t)(q % R);
      sl.nprime[q] = nb[(int64_t)r * E + sl.dexp[d]];
    }
    for (int64_t s = tid; s < S; s += kSchThreads) {
      const int32_t e = se[s];
      sl.Ap[s] = e >= 0 ? sa[s] : 0;
      sl.dsl[s] = e >= 0 ? sl.dmap[e] : -1;
      sl.need[s] = 1;
      sl.bid[s] = -1;
    }
    for (int32_t r = tid; r < R; r += kSchThreads) {
      price[r] = 0.0;
      rkey[r] = 0;
      rwin[r] = INT_MAX;
      served[r] = 0;
    }
    __syncthreads();

    const int64_t tmax = p.t_max > 0 ? p.t_max : S * (R + 1);
    int64_t rounds = 0;
    for (int64_t t = 1; t <= tmax; ++t) {
      // (a) slots whose bid must be recomputed
      int32_t nw = 0;
      for (int64_t base = 0; base < S; base += kSchThreads) {
        const int64_t s = base + tid;
        const bool f = s < S && sl.Ap[s] > 0 && sl.dsl[s] >= 0 && sl.need[s];
        int32_t tot;
        const int32_t pos = compact_pos(f, wave_cnt, tot);
        if (f) sl.work[nw + pos] = (int32_t)s;
        nw += tot;
      }
      // one wave per slot: argmax over ranks r with tokens of the slot's expert
      // of Bauct[r][host] - price[r], lowest r on ties
      for (int32_t w = wid; w < nw; w += kSchWaves) {
        const int32_t s = sl.work[w];
        const int32_t host = s / K;
        const int32_t* np_ = sl.nprime + (int64_t)sl.dsl[s] * R;
        double bs = -INFINITY;
        int32_t br = INT_MAX;
        for (int32_t r = lane; r < R; r += kWave) {
          if (np_[r] <= 0) continue;
          const double sc = p.Bauct[(int64_t)r * R + host] - price[r];
          if (sc > bs) { bs = sc; br = r; }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
          const double os = __shfl_xor(bs, o, kWave);
          const int32_t orr = __shfl_xor(br, o, kWave);
          if (os > bs || (os == bs && orr < br)) { bs = os; br = orr; }
        }
        if (lane == 0) {
          sl.bid[s] = br == INT_MAX ? -1 : br;
          sl.bid_s[s] = bs;
          sl.need[s] = 0;
        }
      }
      __syncthreads();
      // (b) each rank keeps its best bidder: max score, then lowest slot
      bool any = false;
      for (int64_t s = tid; s < S; s += kSchThreads) {
        if (sl.Ap[s] > 0 && sl.bid[s] >= 0) {
          atomicMax(reinterpret_cast<unsigned long long*>(&rkey[sl.bid[s]]),
                    (unsigned long long)auction_key(sl.bid_s[s]));
          any = true;
        }
      }
      if (!block_any(any, wave_cnt)) break;  // no bid: the state is final
      for (int64_t s = tid; s < S; s += kSchThreads) {
        if (sl.Ap[s] > 0 && sl.bid[s] >= 0 && auction_key(sl.bid_s[s]) == rkey[sl.bid[s]])
          atomicMin(&rwin[sl.bid[s]], (int32_t)s);
      }
      __syncthreads();
      // (c) transfers; a rank that moved tokens raises its price
      for (int32_t r = tid; r < R; r += kSchThreads) {
        const int32_t s = rwin[r];
        int32_t did = 0;
        if (s != INT_MAX) {
          int32_t* np_ = sl.nprime + (int64_t)sl.dsl[s] * R + r;
          const int64_t have = *np_;
          const int64_t x = have < sl.Ap[s] ? have : sl.Ap[s];
          Xb[(int64_t)r * S + s] += (int32_t)x;
          *np_ -= (int32_t)x;
          sl.Ap[s] -= x;
          if (x > 0) price[r] = price[r] + p.price_step;
          did = 1;
        }
        served[r] = did;
        rkey[r] = 0;
        rwin[r] = INT_MAX;
      }
      __syncthreads();
      // (d) a slot re-bids if its rank served or ran out of the slot's expert
      for (int64_t s = tid; s < S; s += kSchThreads) {
        const int32_t r = sl.bid[s];
        if (sl.Ap[s] > 0 && r >= 0 && (served[r] || sl.nprime[(int64_t)sl.dsl[s] * R + r] <= 0))
          sl.need[s] = 1;
      }
      __syncthreads();
      rounds = t;
    }

    // ---- outputs -----------------------------------------------------------------
    __shared__ int64_t red[kSchWaves];
    int64_t left = 0;
    for (int64_t s = tid; s < S; s += kSchThreads) left += sl.Ap[s];
    left = wave_sum_i64(left);
    if (lane == 0) red[wid] = left;
    __syncthreads();
    if (tid == 0) {
      int64_t tot = 0;
      for (int w = 0; w < kSchWaves; ++w) tot += red[w];
      p.unfilled[b] = tot;
      if (p.rounds_used) { p.rounds_used[2 * b] = used2; p.rounds_used[2 * b + 1] = (int32_t)rounds; }
      if (p.status) p.status[b] = tot > 0 ? TAOT_ST_UNFILLED : 0u;
    }
    __syncthreads();
  }
}


// ===========================================================================
// One-wave path.  Same arithmetic and order as schedule_kernel, with all
// per-problem state in LDS, one 64-lane wave per problem and no block
// barriers.  It serves R <= 256 and needs every column of Bauct to take few
// distinct values (as topology costs do):
//
// Phase-3 bids by tiers.  The ranks of host column h split into tiers of equal
// bonus (descending).  With prices that start at 0 and rise by a fixed step on
// each service, a rank's price is a function of its service count, and when
// the step is large against the spacing of doubles at the magnitudes reached,
// bonus - price falls strictly with every service.  Within a tier the argmax
// of the score is then the lowest-index rank among those with the fewest
// services, found with a bit-sliced minimum over the count bit-planes; the
// bid is the best tier result under (max score, lowest rank), and tiers whose
// bonus is below the best score so far are skipped (price >= 0).  A price step
// of 0 keeps every price at 0, and the argmax is the lowest rank of the first
// non-empty tier.  A prepass checks the conditions on the device and sends
// problems to schedule_kernel when they fail, as it does problems whose
// candidate or slot-expert counts exceed the LDS layout.

constexpr int kDistinctCap = 64;   // distinct slot experts per problem in LDS
constexpr int kTierMax = 4;        // distinct bonus values per host column
constexpr int kTierWords = 4;      // 64-rank words of a rank set (R <= 256)
constexpr int kStructCap = 32;     // distinct host tier structures kept in LDS
constexpr int kPlanes = 17;        // count bit-planes: counts <= R*K <= 65536

// Tier structure of column h of Bauct: its distinct bonuses in descending
// order and the rank set of each; ntier[h] = -1 if there are more than
// kTierMax.  NaN and -inf bonuses never win a bid and belong to no tier.
__global__ void __launch_bounds__(256)
auction_tiers_kernel(const double* __restrict__ Bauct, int32_t R, int32_t* __restrict__ ntier,
                     double* __restrict__ tv, uint64_t* __restrict__ tmask) {
  __shared__ double vals[kTierMax];
  __shared__ int32_t nv;
  __shared__ unsigned long long msk[kTierMax * kTierWords];
  const int32_t h = blockIdx.x, tid = threadIdx.x;
  if (tid < kTierMax * kTierWords) msk[tid] = 0ull;
  if (tid == 0) {
    int32_t n = 0;
    for (int32_t r = 0; r < R && n >= 0; ++r) {
      const double v = Bauct[(int64_t)r * R + h];
      if (v != v || v == -INFINITY) continue;
      int32_t pos = 0;
      bool dup = false;
      for (int32_t i = 0; i < n; ++i) {
        dup |= vals[i] == v;
        pos += vals[i] > v;
      }
      if (dup) continue;
      if (n == kTierMax) { n = -1; break; }
      for (int32_t i = n; i > pos; --i) vals[i] = vals[i - 1];
      vals[pos] = v;
      ++n;
    }
    nv = n;
  }
  __syncthreads();
  const int32_t n = nv;
  for (int32_t r = tid; r < R && n > 0; r += blockDim.x) {
    const double v = Bauct[(int64_t)r * R + h];
    for (int32_t i = 0; i < n; ++i)
      if (vals[i] == v) atomicOr(&msk[i * kTierWords + (r >> 6)], 1ull << (r & 63));
  }
  __syncthreads();
  if (tid == 0) ntier[h] = n;
  if (tid < kTierMax) tv[(int64_t)h * kTierMax + tid] = tid < n ? vals[tid] : -INFINITY;
  if (tid < kTierMax * kTierWords)
    tmask[(int64_t)h * kTierMax * kTierWords + tid] = tid / kTierWords < n ? msk[tid] : 0ull;
}

// Deduplicates the host tier structures into a table of at most kStructCap
// (one block, one thread per host): sidx[h] is host h's entry, hdr[0] the
// table size, hdr[1] = 1 when the tier search is exact for this Bauct and
// price step: every column has at most kTierMax values, none is +inf, the
// table fits, and the step is 0 or exceeds twice the spacing of doubles at
// max|bonus| + S * step (prices stay below S * step: a rank serves each slot
// at most once).
__global__ void __launch_bounds__(256)
auction_struct_kernel(const int32_t* __restrict__ ntier, const double* __restrict__ tv,
                      const uint64_t* __restrict__ tmask, int32_t R, int64_t S, double step,
                      int32_t* __restrict__ sidx, int32_t* __restrict__ cn, double* __restrict__ cv,
                      uint64_t* __restrict__ cm, int32_t* __restrict__ hdr) {
  __shared__ int32_t first[256];
  const int32_t h = threadIdx.x;
  constexpr int kRow = kTierMax * kTierWords;
  if (h < R) {
    const int32_t nh = ntier[h];
    int32_t f = h;
    for (int32_t g = 0; g < h && f == h; ++g) {
      bool eq = ntier[g] == nh;
      for (int32_t t = 0; t < kTierMax && eq; ++t) eq = tv[g * kTierMax + t] == tv[h * kTierMax + t];
      for (int32_t q = 0; q < kRow && eq; ++q) eq = tmask[g * kRow + q] == tmask[h * kRow + q];
      if (eq) f = g;
    }
    first[h] = f;
  }
  __syncthreads();
  if (h == 0) {
    int32_t ns = 0;
    double vm = 0.0;
    bool ok = true;
    for (int32_t g = 0; g < R; ++g) {
      ok &= ntier[g] >= 0;
      if (first[g] != g) {
        sidx[g] = sidx[first[g]];
        continue;
      }
      for (int32_t t = 0; t < kTierMax; ++t) {
        const double v = tv[g * kTierMax + t];
        if (t < ntier[g]) {
          ok &= v != INFINITY;
          vm = fmax(vm, fabs(v));
        }
      }
      if (ns < kStructCap) {
        cn[ns] = ntier[g] > 0 ? ntier[g] : 0;
        for (int32_t t = 0; t < kTierMax; ++t) cv[ns * kTierMax + t] = tv[g * kTierMax + t];
        for (int32_t q = 0; q < kRow; ++q) cm[ns * kRow + q] = tmask[g * kRow + q];
      }
      sidx[g] = ns;
      ++ns;
    }
    ok &= ns <= kStructCap;
    const double top = vm + (double)S * step * 1.01 + 1.0;
    ok &= step == 0.0 || (step > 0.0 && step > 2.0 * (nextafter(top, INFINITY) - top));
    hdr[0] = ns < kStructCap ? ns : kStructCap;
    hdr[1] = ok ? 1 : 0;
  }
}

struct WaveLds {
  // both phases
  int32_t* slot_ec;   // [S] candidate index of the slot's expert or -1
  int32_t* amt;       // [S] phase 2: slot amount; phase 3: tokens still planned
  int32_t* ce;        // [NEC] candidate experts (spill > 0), ascending
  // phase 2
  int32_t* cr; int64_t* spare_p; int32_t* matched; int32_t* prop_e; double* prop_s; int32_t* assigned;
  int64_t* spill_p; uint64_t* ekey; int32_t* ewin;
  // phase 3 (aliases the phase-2 region)
  double* price; uint64_t* rkey; int32_t* rwin; uint64_t* served;
  int32_t* bid; double* bid_s; int32_t* dsl; int32_t* work;
  uint64_t* vmask; int32_t* dexp; int32_t* dmap;
  int32_t* cnt; uint64_t* planes;
  int32_t* sidx; int32_t* cn; double* cv; uint64_t* cm;
  size_t bytes;
};

__host__ __device__ inline WaveLds carve_wave(char* base, int32_t R, int32_t K, int32_t NEC) {
  WaveLds w;
  const int64_t S = (int64_t)R * K;
  const size_t S1 = S > 0 ? (size_t)S : 1;
  const int32_t W64 = (R + 63) / 64;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* q = base + off;
    off = (off + bytes + 15) & ~(size_t)15;
    return q;
  };
  w.slot_ec = (int32_t*)take(4 * S1);
  w.amt = (int32_t*)take(4 * S1);
  w.ce = (int32_t*)take(4 * (size_t)NEC);
  const size_t split = off;
  w.cr = (int32_t*)take(4 * (size_t)R); w.spare_p = (int64_t*)take(8 * (size_t)R);
  w.matched = (int32_t*)take(4 * (size_t)R); w.prop_e = (int32_t*)take(4 * (size_t)R);
  w.prop_s = (double*)take(8 * (size_t)R); w.assigned = (int32_t*)take(4 * (size_t)R * (K > 0 ? K : 1));
  w.spill_p = (int64_t*)take(8 * (size_t)NEC); w.ekey = (uint64_t*)take(8 * (size_t)NEC);
  w.ewin = (int32_t*)take(4 * (size_t)NEC);
  const size_t end2 = off;
  off = split;
  w.price = (double*)take(8 * (size_t)R); w.rkey = (uint64_t*)take(8 * (size_t)R);
  w.rwin = (int32_t*)take(4 * (size_t)R); w.served = (uint64_t*)take(8 * (size_t)W64);
  w.bid = (int32_t*)take(4 * S1); w.bid_s = (double*)take(8 * S1);
  w.dsl = (int32_t*)take(4 * S1); w.work = (int32_t*)take(4 * S1);
  w.vmask = (uint64_t*)take(8 * (size_t)kDistinctCap * kTierWords);
  w.dexp = (int32_t*)take(4 * kDistinctCap); w.dmap = (int32_t*)take(4 * (size_t)NEC);
  w.cnt = (int32_t*)take(4 * (size_t)R); w.planes = (uint64_t*)take(8 * kPlanes * kTierWords);
  w.sidx = (int32_t*)take(4 * (size_t)R); w.cn = (int32_t*)take(4 * kStructCap);
  w.cv = (double*)take(8 * kStructCap * kTierMax);
  w.cm = (uint64_t*)take(8 * kStructCap * kTierMax * kTierWords);
  w.bytes = end2 > off ? end2 : off;
  return w;
}

struct WaveParams {
  SchParams s;
  const int32_t* sidx;   // [R] host -> tier structure
  const int32_t* cn;     // [kStructCap] tiers per structure
  const double* cv;      // [kStructCap][kTierMax] tier bonuses, descending
  const uint64_t* cm;    // [kStructCap][kTierMax][kTierWords] tier rank sets
  const int32_t* hdr;    // [0] structures, [1] tier search exact
  int32_t* fallback;     // [B] 1 = left to schedule_kernel
  int32_t* nprime;       // [B][kDistinctCap][R]
  int32_t NEC;           // candidate-expert capacity of the LDS layout
};

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
}

__device__ __forceinline__ int32_t wave_max_i32(int32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const int32_t u = __shfl_xor(v, o, kWave);
    v = u > v ? u : v;
  }
  return __builtin_amdgcn_readfirstlane(v);
}

__global__ void __launch_bounds__(kWave) schedule_wave_kernel(WaveParams wp) {
  extern __shared__ __attribute__((aligned(16))) char wlds[];
  const SchParams& p = wp.s;
  const int lane = threadIdx.x;
  const int64_t b = blockIdx.x;
  const int32_t R = p.R, E = p.E, K = p.K;
  const int64_t S = (int64_t)R * K;
  const int32_t W64 = (R + 63) / 64;
  const uint64_t below = (1ull << lane) - 1ull;
  WaveLds L = carve_wave(wlds, R, K, wp.NEC);

  if (wp.hdr[1] == 0) {  // the tier search would not be exact for this Bauct and step
    if (lane == 0) wp.fallback[b] = 1;
    return;
  }
  const int64_t* spill = p.spill + b * E;
  const int64_t* spare = p.spare + b * R;
  const int64_t* excess = p.excess + b * R;
  const float* Tb = p.T + b * (int64_t)R * R;
  int32_t* se = p.slot_expert + b * S;
  int64_t* sa = p.slot_amount + b * S;
  int32_t* Xb = p.X + b * (int64_t)R * S;
  const double alpha = p.alpha[b];
  const double a2 = 0.1 * alpha;

  // ---- validation, candidates, cold ranks ------------------------------------------
  bool badh = false;
  for (int32_t e = lane; e < E; e += kWave) {
    const int32_t h = p.home[e];
    badh |= h < 0 || h >= R;
  }
  if (__ballot(badh) != 0) {
    for (int64_t s = lane; s < S; s += kWave) { se[s] = -1; sa[s] = 0; }
    for (int64_t q = lane; q < (int64_t)R * S; q += kWave) Xb[q] = 0;
    if (lane == 0) {
      p.unfilled[b] = 0;
      if (p.rounds_used) { p.rounds_used[2 * b] = 0; p.rounds_used[2 * b + 1] = 0; }
      if (p.status) p.status[b] = TAOT_ST_BAD_INPUT;
      wp.fallback[b] = 0;
    }
    return;
  }
  int32_t ne = 0, nc = 0;
  int64_t mass = 0;  // bounds every slot amount and transfer
  for (int32_t base = 0; base < E; base += kWave) {
    const int32_t e = base + lane;
    const int64_t v = e < E ? spill[e] : 0;
    const bool f = v > 0;
    const uint64_t m = __ballot(f);
    const int32_t pos = ne + __popcll(m & below);
    if (f && pos < wp.NEC) { L.ce[pos] = e; L.spill_p[pos] = v; }
    ne += __popcll(m);
    mass += f ? v : 0;
  }
  mass = wave_sum_i64(mass);
  if (ne > wp.NEC || mass > INT_MAX) {  // beyond the LDS layout or its 32-bit amounts
    if (lane == 0) wp.fallback[b] = 1;
    return;
  }
  for (int32_t base = 0; base < R; base += kWave) {
    const int32_t r = base + lane;
    const bool f = r < R && spare[r] > 0;
    const uint64_t m = __ballot(f);
    const int32_t pos = nc + __popcll(m & below);
    if (f) { L.cr[pos] = r; L.spare_p[pos] = spare[r]; }
    nc += __popcll(m);
  }
  for (int64_t q = lane; q < (int64_t)nc * K; q += kWave) L.assigned[q] = -1;
  for (int32_t ec = lane; ec < ne; ec += kWave) { L.ekey[ec] = 0; L.ewin[ec] = INT_MAX; }
  for (int64_t s = lane; s < S; s += kWave) { L.slot_ec[s] = -1; L.amt[s] = 0; se[s] = -1; }
  wave_sync();

  // ---- Phase 2: column-priority iterative matching ---------------------------------
  int32_t used2 = 0;
  for (int32_t k = 0; k < K; ++k) {
    for (int32_t rc = lane; rc < nc; rc += kWave) L.matched[rc] = 0;
    wave_sync();
    for (int32_t inner = 0; inner < nc; ++inner) {
      bool proposed = false;
      for (int32_t rc = lane; rc < nc; rc += kWave) {
        int32_t best = -1;
        double bs = -INFINITY;
        const int64_t sp = L.spare_p[rc];
        if (!L.matched[rc] && sp > 0) {
          const int32_t r = L.cr[rc];
          for (int32_t ec = 0; ec < ne; ++ec) {
            const int64_t spl = L.spill_p[ec];
            if (spl <= 0) continue;
            const int32_t h = p.home[L.ce[ec]];
            if (h == r) continue;
            bool taken = false;
            for (int32_t kk = 0; kk < k; ++kk) taken |= L.assigned[(int64_t)rc * K + kk] == ec;
            if (taken) continue;
            const double q = (double)(spl < sp ? spl : sp);
            const double t1 = alpha * p.Bpref[(int64_t)h * R + r];
            const double ex = (double)excess[h];
            const double tn = (double)Tb[(int64_t)h * R + r] / (ex > kEps0 ? ex : kEps0);
            const double t2 = a2 * tn;
            const double score = (q + t1) + t2;
            if (score > bs) { bs = score; best = ec; }
          }
        }
        L.prop_e[rc] = best;
        L.prop_s[rc] = bs;
        proposed |= best >= 0;
      }
      if (__ballot(proposed) == 0) break;  // nothing can change any more
      wave_sync();
      // each proposed expert keeps its best proposer: max score, then lowest rank
      for (int32_t rc = lane; rc < nc; rc += kWave)
        if (L.prop_e[rc] >= 0)
          atomicMax(reinterpret_cast<unsigned long long*>(&L.ekey[L.prop_e[rc]]),
                    (unsigned long long)ordered_key(L.prop_s[rc]));
      wave_sync();
      for (int32_t rc = lane; rc < nc; rc += kWave)
        if (L.prop_e[rc] >= 0 && ordered_key(L.prop_s[rc]) == L.ekey[L.prop_e[rc]])
          atomicMin(&L.ewin[L.prop_e[rc]], rc);
      wave_sync();
      // winners take g = min(spill, spare) into slot k of their rank
      for (int32_t ec = lane; ec < ne; ec += kWave) {
        const int32_t w = L.ewin[ec];
        if (w != INT_MAX) {
          const int64_t g = L.spill_p[ec] < L.spare_p[w] ? L.spill_p[ec] : L.spare_p[w];
          L.spill_p[ec] -= g;
          L.spare_p[w] -= g;
          L.matched[w] = 1;
          L.assigned[(int64_t)w * K + k] = ec;
          const int64_t s = (int64_t)L.cr[w] * K + k;
          L.slot_ec[s] = ec;
          L.amt[s] += (int32_t)g;
          se[s] = L.ce[ec];
        }
        L.ekey[ec] = 0;
        L.ewin[ec] = INT_MAX;
      }
      wave_sync();
      ++used2;
    }
  }
  for (int64_t s = lane; s < S; s += kWave) sa[s] = L.amt[s];

  // ---- Phase 3: Lagrangian auction ---------------------------------------------------
  // distinct slot experts, in ascending candidate (= expert) order
  for (int32_t ec = lane; ec < ne; ec += kWave) L.dmap[ec] = 0;
  wave_sync();
  for (int64_t s = lane; s < S; s += kWave)
    if (L.slot_ec[s] >= 0) L.dmap[L.slot_ec[s]] = 1;
  wave_sync();
  int32_t D = 0;
  for (int32_t base = 0; base < ne; base += kWave) {
    const int32_t ec = base + lane;
    const bool f = ec < ne && L.dmap[ec] == 1;
    const uint64_t m = __ballot(f);
    const int32_t pos = D + __popcll(m & below);
    if (ec < ne) L.dmap[ec] = f ? pos : -1;
    if (f && pos < kDistinctCap) L.dexp[pos] = L.ce[ec];
    D += __popcll(m);
  }
  if (D > kDistinctCap) {
    if (lane == 0) wp.fallback[b] = 1;
    return;
  }
  wave_sync();
  // tokens of each slot expert per rank (device memory) and the valid-rank sets
  int32_t* np = wp.nprime + b * (int64_t)kDistinctCap * R;
  const int32_t* nb = p.n + b * (int64_t)R * E;
  for (int32_t d = 0; d < D; ++d) {
    const int32_t e = L.dexp[d];
    for (int32_t w = 0; w < kTierWords; ++w) {
      const int32_t r = w * kWave + lane;
      const int32_t v = r < R ? nb[(int64_t)r * E + e] : 0;
      if (r < R) np[(int64_t)d * R + r] = v;
      const uint64_t m = __ballot(v > 0);
      if (lane == 0) L.vmask[d * kTierWords + w] = m;
    }
  }
  // slots that bid in the first round
  int32_t nwork = 0;
  for (int64_t base = 0; base < S; base += kWave) {
    const int64_t s = base + lane;
    const int32_t ec = s < S ? L.slot_ec[s] : -1;
    if (s < S) {
      L.dsl[s] = ec >= 0 ? L.dmap[ec] : -1;
      L.bid[s] = -1;
      if (ec < 0) L.amt[s] = 0;
    }
    const bool f = ec >= 0 && L.amt[s] > 0;
    const uint64_t m = __ballot(f);
    if (f) L.work[nwork + __popcll(m & below)] = (int32_t)s;
    nwork += __popcll(m);
  }
  for (int32_t r = lane; r < R; r += kWave) {
    L.price[r] = 0.0;
    L.rkey[r] = 0;
    L.rwin[r] = INT_MAX;
    L.cnt[r] = 0;
    L.sidx[r] = wp.sidx[r];
  }
  for (int32_t q = lane; q < kPlanes * kTierWords; q += kWave) L.planes[q] = 0ull;
  const int32_t ns = wp.hdr[0];
  for (int32_t q = lane; q < ns; q += kWave) L.cn[q] = wp.cn[q];
  for (int32_t q = lane; q < ns * kTierMax; q += kWave) L.cv[q] = wp.cv[q];
  for (int32_t q = lane; q < ns * kTierMax * kTierWords; q += kWave) L.cm[q] = wp.cm[q];
  // X starts at zero; every (rank, slot) pair is served at most once (after a
  // transfer either the rank holds no more tokens of the slot's expert or the
  // slot is full), so transfers below are plain stores
  {
    int4* x4 = reinterpret_cast<int4*>(Xb);
    const int64_t n4 = ((int64_t)R * S) / 4;
    if ((reinterpret_cast<uintptr_t>(Xb) & 15u) == 0) {
      for (int64_t q = lane; q < n4; q += kWave) x4[q] = make_int4(0, 0, 0, 0);
      for (int64_t q = n4 * 4 + lane; q < (int64_t)R * S; q += kWave) Xb[q] = 0;
    } else {
      for (int64_t q = lane; q < (int64_t)R * S; q += kWave) Xb[q] = 0;
    }
  }
  wave_sync();

  const double step = p.price_step;
  const bool track = step > 0.0;  // counts order the prices; with step 0 all prices stay 0
  int32_t maxc = 0;               // largest service count so far
  const int64_t tmax = p.t_max > 0 ? p.t_max : S * (R + 1);
  int64_t rounds = 0;
  for (int64_t t = 1; t <= tmax; ++t) {
    // (a) bids of the listed slots: argmax over ranks holding tokens of the
    //     slot's expert of Bauct[r][host] - price[r], lowest rank on ties
    const int32_t nplanes = maxc > 0 ? 32 - __builtin_clz((uint32_t)maxc) : 0;
    for (int32_t w0 = 0; w0 < nwork; w0 += kWave) {
      if (w0 + lane >= nwork) continue;
      const int32_t s = L.work[w0 + lane];
      const int32_t host = s / K;
      const uint64_t* vm = L.vmask + L.dsl[s] * kTierWords;
      const int32_t st = L.sidx[host];
      const int32_t nt = L.cn[st];
      uint64_t valid[kTierWords];
#pragma unroll
      for (int w = 0; w < kTierWords; ++w) valid[w] = vm[w];
      double bs = -INFINITY;
      int32_t br = INT_MAX;
      for (int32_t ti = 0; ti < nt; ++ti) {
        const double v = L.cv[st * kTierMax + ti];
        if (v < bs) break;  // every score in this tier and the next is <= v
        const uint64_t* tm = L.cm + (st * kTierMax + ti) * kTierWords;
        uint64_t c[kTierWords];
        uint64_t any = 0;
#pragma unroll
        for (int w = 0; w < kTierWords; ++w) { c[w] = tm[w] & valid[w]; any |= c[w]; }
        if (!any) continue;
        // fewest services: keep the ranks with a 0 in each bit-plane, top down,
        // whenever any remain
        for (int32_t j = nplanes - 1; j >= 0; --j) {
          uint64_t m[kTierWords];
          uint64_t mm = 0;
#pragma unroll
          for (int w = 0; w < kTierWords; ++w) { m[w] = c[w] & ~L.planes[j * kTierWords + w]; mm |= m[w]; }
          if (mm) {
#pragma unroll
            for (int w = 0; w < kTierWords; ++w) c[w] = m[w];
          }
        }
        int32_t r = INT_MAX;
#pragma unroll
        for (int w = kTierWords - 1; w >= 0; --w)
          if (c[w]) r = w * kWave + __builtin_ctzll(c[w]);
        const double sc = v - L.price[r];
        if (sc > bs || (sc == bs && r < br)) { bs = sc; br = r; }
      }
      L.bid[s] = br == INT_MAX ? -1 : br;
      L.bid_s[s] = bs;
    }
    wave_sync();
    // (b) each rank keeps its best bidder: max score, then lowest slot
    bool any = false;
    for (int64_t s = lane; s < S; s += kWave) {
      const int32_t r = L.bid[s];
      if (L.amt[s] > 0 && r >= 0) {
        atomicMax(reinterpret_cast<unsigned long long*>(&L.rkey[r]),
                  (unsigned long long)auction_key(L.bid_s[s]));
        any = true;
      }
    }
    if (__ballot(any) == 0) break;  // no bid: the state is final
    wave_sync();
    for (int64_t s = lane; s < S; s += kWave) {
      const int32_t r = L.bid[s];
      if (L.amt[s] > 0 && r >= 0 && auction_key(L.bid_s[s]) == L.rkey[r]) atomicMin(&L.rwin[r], (int32_t)s);
    }
    wave_sync();
    // (c) transfers; a rank that moved tokens raises its price
    int32_t newmax = 0;
    for (int32_t w = 0; w < W64; ++w) {
      const int32_t r = w * kWave + lane;
      bool did = false;
      if (r < R) {
        const int32_t s = L.rwin[r];
        if (s != INT_MAX) {
          const int32_t d = L.dsl[s];
          int32_t* cell = np + (int64_t)d * R + r;
          const int32_t have = *cell;
          const int32_t x = have < L.amt[s] ? have : L.amt[s];
          Xb[(int64_t)r * S + s] = x;
          *cell = have - x;
          L.amt[s] -= x;
          if (x > 0) {
            L.price[r] = L.price[r] + step;
            if (track) {
              const int32_t c0 = L.cnt[r], c1 = c0 + 1;
              L.cnt[r] = c1;
              newmax = c1 > newmax ? c1 : newmax;
              for (uint32_t flip = (uint32_t)(c0 ^ c1); flip; flip &= flip - 1)
                atomicXor(reinterpret_cast<unsigned long long*>(
                              &L.planes[__builtin_ctz(flip) * kTierWords + w]),
                          1ull << lane);
            }
          }
          if (have - x <= 0)
            atomicAnd(reinterpret_cast<unsigned long long*>(&L.vmask[d * kTierWords + w]), ~(1ull << lane));
          did = true;
        }
        L.rkey[r] = 0;
        L.rwin[r] = INT_MAX;
      }
      const uint64_t m = __ballot(did);
      if (lane == 0) L.served[w] = m;
    }
    const int32_t m2 = wave_max_i32(newmax);
    maxc = m2 > maxc ? m2 : maxc;
    wave_sync();
    // (d) a slot re-bids if its rank served or ran out of the slot's expert
    nwork = 0;
    for (int64_t base = 0; base < S; base += kWave) {
      const int64_t s = base + lane;
      bool f = false;
      if (s < S) {
        const int32_t r = L.bid[s];
        if (L.amt[s] > 0 && r >= 0) {
          const bool served = (L.served[r >> 6] >> (r & 63)) & 1ull;
          const bool valid = (L.vmask[L.dsl[s] * kTierWords + (r >> 6)] >> (r & 63)) & 1ull;
          f = served || !valid;
        }
      }
      const uint64_t m = __ballot(f);
      if (f) L.work[nwork + __popcll(m & below)] = (int32_t)s;
      nwork += __popcll(m);
    }
    wave_sync();
    rounds = t;
  }

  int64_t left = 0;
  for (int64_t s = lane; s < S; s += kWave) left += L.amt[s];
  left = wave_sum_i64(left);
  if (lane == 0) {
    p.unfilled[b] = left;
    if (p.rounds_used) { p.rounds_used[2 * b] = used2; p.rounds_used[2 * b + 1] = (int32_t)rounds; }
    if (p.status) p.status[b] = left > 0 ? TAOT_ST_UNFILLED : 0u;
    wp.fallback[b] = 0;
  }
}
}  // namespace

static int32_t sched_grid(int32_t B) { return B < kSchMaxGrid ? B : kSchMaxGrid; }

namespace {

struct SchWs {
  char* slab;          // general path: one slab per resident workgroup
  int32_t* fallback;   // [B]
  int32_t* ntier;      // [R]
  double* tv;          // [R][kTierMax]
  uint64_t* tmask;     // [R][kTierMax][kTierWords]
  int32_t* sidx;       // [R]
  int32_t* cn;         // [kStructCap]
  double* cv;          // [kStructCap][kTierMax]
  uint64_t* cm;        // [kStructCap][kTierMax][kTierWords]
  int32_t* hdr;        // [2]
  int32_t* nprime;     // [B][kDistinctCap][R]
  int64_t slab_bytes;
  size_t bytes;
};

SchWs carve_sched(void* ws, int32_t B, int32_t R, int32_t E, int32_t K) {
  Carver c{static_cast<char*>(ws)};
  SchWs w;
  w.slab_bytes = round_up((int64_t)carve_slab(nullptr, R, E, K).bytes, 256);
  w.slab = c.take<char>((size_t)w.slab_bytes * (B > 0 ? sched_grid(B) : 0));
  w.fallback = c.take<int32_t>((size_t)B);
  w.ntier = c.take<int32_t>((size_t)R);
  w.tv = c.take<double>((size_t)R * kTierMax);
  w.tmask = c.take<uint64_t>((size_t)R * kTierMax * kTierWords);
  w.sidx = c.take<int32_t>((size_t)R);
  w.cn = c.take<int32_t>(kStructCap);
  w.cv = c.take<double>(kStructCap * kTierMax);
  w.cm = c.take<uint64_t>(kStructCap * kTierMax * kTierWords);
  w.hdr = c.take<int32_t>(2);
  w.nprime = c.take<int32_t>((size_t)B * kDistinctCap * R);
  w.bytes = c.off;
  return w;
}

constexpr size_t kWaveLdsMax = 64 * 1024;  // keep several problems resident per CU

}  // namespace

size_t schedule_ws(int32_t B, int32_t R, int32_t E, int32_t K) { return carve_sched(nullptr, B, R, E, K).bytes; }

taot_status launch_schedule(const int32_t* n, const int64_t* spill, const int64_t* spare,
                            const int64_t* excess, const double* alpha, const int32_t* home,
                            const float* T, const double* Bpref, const double* Bauct, int32_t B,
                            int32_t R, int32_t E, int32_t K, double price_step, int64_t t_max,
                            int32_t* slot_expert, int64_t* slot_amount, int32_t* X,
                            int64_t* unfilled, int32_t* rounds_used, uint32_t* status, void* ws,
                            hipStream_t stream) {
  if (B == 0) return TAOT_OK;
  SchWs w = carve_sched(ws, B, R, E, K);
  SchParams p{n, spill, spare, excess, alpha, home, T, Bpref, Bauct, B, R, E, K, price_step, t_max,
              slot_expert, slot_amount, X, unfilled, rounds_used, status, w.slab, w.slab_bytes, w.fallback};
  // one-wave path when its LDS layout fits
  const int32_t NEC = E < 512 ? E : 512;
  const int64_t S = (int64_t)R * K;
  const size_t wlds = carve_wave(nullptr, R, K, NEC).bytes;
  const bool wave_ok = R <= kTierWords * kWave && S > 0 && S <= 65536 && wlds <= kWaveLdsMax;
  if (wave_ok) {
    hipLaunchKernelGGL(auction_tiers_kernel, dim3((unsigned)R), dim3(256), 0, stream, Bauct, R, w.ntier, w.tv,
                       w.tmask);
    if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
    hipLaunchKernelGGL(auction_struct_kernel, dim3(1), dim3(256), 0, stream, w.ntier, w.tv, w.tmask, R, S,
                       price_step, w.sidx, w.cn, w.cv, w.cm, w.hdr);
    if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
    WaveParams wp{p, w.sidx, w.cn, w.cv, w.cm, w.hdr, w.fallback, w.nprime, NEC};
    hipLaunchKernelGGL(schedule_wave_kernel, dim3((unsigned)B), dim3(kWave), wlds, stream, wp);
    if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  } else {
    p.fallback = nullptr;  // the general kernel takes every problem
  }
  const size_t lds = (size_t)R * (sizeof(double) + sizeof(uint64_t) + 2 * sizeof(int32_t));
  if (lds > 65536 && hipFuncSetAttribute((const void*)schedule_kernel,
                                         hipFuncAttributeMaxDynamicSharedMemorySize,
                                         (int)lds) != hipSuccess)
    return TAOT_ERR_LAUNCH;
  hipLaunchKernelGGL(schedule_kernel, dim3((unsigned)sched_grid(B)), dim3(kSchThreads), lds, stream, p);
  return hipGetLastError() == hipSuccess ? TAOT_OK : TAOT_ERR_LAUNCH;
}

}  // namespace taot
