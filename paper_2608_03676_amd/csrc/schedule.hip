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

}  // namespace

static int32_t sched_grid(int32_t B) { return B < kSchMaxGrid ? B : kSchMaxGrid; }

size_t schedule_ws(int32_t B, int32_t R, int32_t E, int32_t K) {
  const size_t slab = (size_t)round_up((int64_t)carve_slab(nullptr, R, E, K).bytes, 256);
  return slab * (size_t)(B > 0 ? sched_grid(B) : 0);
}

taot_status launch_schedule(const int32_t* n, const int64_t* spill, const int64_t* spare,
                            const int64_t* excess, const double* alpha, const int32_t* home,
                            const float* T, const double* Bpref, const double* Bauct, int32_t B,
                            int32_t R, int32_t E, int32_t K, double price_step, int64_t t_max,
                            int32_t* slot_expert, int64_t* slot_amount, int32_t* X,
                            int64_t* unfilled, int32_t* rounds_used, uint32_t* status, void* ws,
                            hipStream_t stream) {
  if (B == 0) return TAOT_OK;
  const int64_t slab = round_up((int64_t)carve_slab(nullptr, R, E, K).bytes, 256);
  SchParams p{n, spill, spare, excess, alpha, home, T, Bpref, Bauct, B, R, E, K, price_step, t_max,
              slot_expert, slot_amount, X, unfilled, rounds_used, status, static_cast<char*>(ws), slab};
  const size_t lds = (size_t)R * (sizeof(double) + sizeof(uint64_t) + 2 * sizeof(int32_t));
  if (lds > 65536 && hipFuncSetAttribute((const void*)schedule_kernel,
                                         hipFuncAttributeMaxDynamicSharedMemorySize,
                                         (int)lds) != hipSuccess)
    return TAOT_ERR_LAUNCH;
  hipLaunchKernelGGL(schedule_kernel, dim3((unsigned)sched_grid(B)), dim3(kSchThreads), lds, stream, p);
  return hipGetLastError() == hipSuccess ? TAOT_OK : TAOT_ERR_LAUNCH;
}

}  // namespace taot
