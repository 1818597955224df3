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
  const int32_t* fallback;  // [B] 1 = the LDS-resident kernel left this problem to us (nullable)
  uint32_t flags;           // TAOT_SCH_*
};

// Weights of the Phase-2 score terms: alpha for alpha * Bpref and 0.1 * alpha
// for the flow hint, or 0 for a term the flags drop (it then enters the sum
// as +0, in the same evaluation order).
__device__ __forceinline__ double topo_weight(uint32_t flags, double alpha) {
  return (flags & TAOT_SCH_NO_TOPO) ? 0.0 : alpha;
}
__device__ __forceinline__ double flow_weight(uint32_t flags, double alpha) {
  return (flags & TAOT_SCH_NO_FLOW) ? 0.0 : 0.1 * alpha;
}

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
  __shared__ double sh_rbs[kSchWaves];  // row-priority argmax, per wave
  __shared__ int32_t sh_rbi[kSchWaves];
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
    const double alpha = topo_weight(p.flags, p.alpha[b]);
    const double a2 = flow_weight(p.flags, p.alpha[b]);  // weight of the OT hint

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
    if (p.flags & TAOT_SCH_ROW_PRIORITY) {
      // the experts-outer greedy (ablation): per slot round, the experts with
      // spill left in order of spill (largest first, lower index on ties), each
      // taking its best ranks one at a time until its spill is gone
      for (int32_t k = 0; k < K; ++k) {
        int32_t nord = 0;
        for (int32_t base = 0; base < ne; base += kSchThreads) {
          const int32_t ec = base + tid;
          const int64_t v = ec < ne ? sl.spill_p[ec] : 0;
          int32_t tot;
          compact_pos(v > 0, wave_cnt, tot);
          if (v > 0) {
            int32_t pos = 0;
            for (int32_t o = 0; o < ne; ++o) {
              const int64_t u = sl.spill_p[o];
              pos += u > v || (u == v && o < ec);
            }
            sl.win[pos] = ec;
          }
          nord += tot;
        }
        __syncthreads();
        for (int32_t i = 0; i < nord; ++i) {
          const int32_t ec = sl.win[i];
          const int32_t h = p.home[sl.ce[ec]];
          for (;;) {
            const int64_t spl = sl.spill_p[ec];
            if (spl <= 0) break;
            double bs = -INFINITY;
            int32_t best = INT_MAX;
            for (int32_t rc = tid; rc < nc; rc += kSchThreads) {
              const int64_t sp = sl.spare_p[rc];
              const int32_t r = sl.cr[rc];
              if (sp <= 0 || r == h || sl.assigned[(int64_t)rc * K + k] >= 0) continue;
              bool taken = false;
              for (int32_t kk = 0; kk < k; ++kk) taken |= sl.assigned[(int64_t)rc * K + kk] == ec;
              if (taken) continue;
              const double q = (double)(spl < sp ? spl : sp);
              const double t1 = alpha * p.Bpref[(int64_t)h * R + r];
              const double ex = (double)excess[h];
              const double tn = (double)Tb[(int64_t)h * R + r] / (ex > kEps0 ? ex : kEps0);
              const double t2 = a2 * tn;
              const double score = (q + t1) + t2;
              if (score > bs) { bs = score; best = rc; }  // rc ascends within a thread
            }
            // block argmax: max score, then lowest cold-rank index (= lowest rank)
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) {
              const double os = __shfl_xor(bs, o, kWave);
              const int32_t oi = __shfl_xor(best, o, kWave);
              if (os > bs || (os == bs && oi < best)) { bs = os; best = oi; }
            }
            if (lane == 0) { sh_rbs[wid] = bs; sh_rbi[wid] = best; }
            __syncthreads();
            if (tid == 0) {
              double b2 = sh_rbs[0];
              int32_t i2 = sh_rbi[0];
              for (int w2 = 1; w2 < kSchWaves; ++w2)
                if (sh_rbs[w2] > b2 || (sh_rbs[w2] == b2 && sh_rbi[w2] < i2)) { b2 = sh_rbs[w2]; i2 = sh_rbi[w2]; }
              if (i2 != INT_MAX) {
                const int64_t g = spl < sl.spare_p[i2] ? spl : sl.spare_p[i2];
                sl.spill_p[ec] -= g;
                sl.spare_p[i2] -= g;
                sl.assigned[(int64_t)i2 * K + k] = ec;
                const int64_t s = (int64_t)sl.cr[i2] * K + k;
                se[s] = sl.ce[ec];
                sa[s] += g;
              }
              sh_flag = i2 != INT_MAX;
            }
            __syncthreads();
            const bool placed = sh_flag != 0;
            __syncthreads();
            if (!placed) break;
            ++used2;
          }
        }
      }
    } else
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
      // the list (in the slab, device memory) is read by other waves below:
      // without this barrier a wave can read an entry of the previous round's
      // list, and a slot that must bid again keeps its old bid for a round
      __syncthreads();
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
// LDS-resident path.  Same arithmetic and order as schedule_kernel, with one
// workgroup per problem and all of its state in LDS and registers.  Two size
// configurations: 256 threads for R <= 256 and R*K <= 1024 (several problems
// per compute unit), 1024 threads for R <= 1024 and R*K <= 4096 (up to
// ~155 KB of LDS, one problem per compute unit).  Both need bonuses (Bauct
// columns) that take few distinct values, as topology costs do.
//
// Phase-3 bids by tiers.  The ranks of host column h split into tiers of equal
// bonus (descending).  With prices that start at 0 and rise by a fixed step on
// each service, a rank's price is a function of its service count, and when
// the step is large against the spacing of doubles at the magnitudes reached,
// bonus - price falls strictly with every service.  Within a tier the argmax
// of the score is then the lowest-index rank among those with the fewest
// services.  Every service raises one count by one and the counts of all
// ranks stay close together, so the kernel keeps them relative to a base
// (the fewest services of any rank): the rank set at the base count, and the
// bit-planes of min(count - base, kRelMax), the relative code.  A tier's
// fewest-services candidate is its lowest rank at the base count when there
// is one, else the lowest rank of the smallest relative code (a bit-sliced
// minimum over the four code planes, words jointly), and when every
// candidate's code is saturated, the bit-sliced minimum over the planes of
// the full counts.  The bid is the best tier result under (max score, lowest
// rank).  No rank's price is below the price P0 of the base count, so a tier
// whose bonus minus P0 is below the best score so far cannot win, nor can any
// later (lower) tier.  A price step of 0 keeps every count and price at 0
// (every rank stays at the base count), and the argmax is the lowest rank of
// the first non-empty tier.
//
// Phase-3 arbitration by bonus.  Every live bid on rank r was placed at r's
// current price (a slot re-bids when its rank serves), so among r's bidders
// the score order is the order of their bonuses when distinct bonuses stay
// distinct after subtracting any reachable price.  A rank's winner is then the
// maximum of the 32-bit key (bonus rank, -slot), taken with one atomicMax.
//
// A prepass checks these conditions on the device and sends problems to
// schedule_kernel when they fail, as it does problems whose candidate or
// slot-expert counts exceed the LDS layout.

constexpr int kTierMax = 4;  // distinct bonus values per host column
constexpr int kRelPlanes = 4;                       // bit-planes of the relative code
constexpr int kRelMax = (1 << kRelPlanes) - 1;      // saturated code: count - base >= kRelMax

struct LdsSmall {
  static constexpr int kT = 256;     // threads per problem
  static constexpr int kTW = 4;      // 64-rank words of a rank set (R <= 256)
  static constexpr int kSC = 32;     // distinct host tier structures in LDS
  static constexpr int kDC = 64;     // distinct slot experts per problem
  static constexpr int kPL = 11;     // count bit-planes: counts <= R*K <= 1024
  static constexpr int kMaxS = 1024; // R*K
  static constexpr int kNEC = 128;   // candidate experts (spill > 0) in LDS
  static constexpr int kWavesPerEU = 8;  // large batches: eight problems per compute unit (20 KB of LDS each at R = 256, K = 2)
};
struct LdsTiny {
  static constexpr int kT = 64;      // one wave per problem: its barriers cost next to nothing
  static constexpr int kTW = 1;      // R <= 64
  static constexpr int kSC = 64;
  static constexpr int kDC = 64;
  static constexpr int kPL = 9;      // counts <= R*K <= 256
  static constexpr int kMaxS = 256;
  static constexpr int kNEC = 128;
  static constexpr int kWavesPerEU = 8;
};
struct LdsLarge {
  static constexpr int kT = 1024;
  static constexpr int kTW = 16;     // R <= 1024
  static constexpr int kSC = 128;
  static constexpr int kDC = 128;
  static constexpr int kPL = 13;     // counts <= R*K <= 4096
  static constexpr int kMaxS = 4096;
  static constexpr int kNEC = 1024;
  static constexpr int kWavesPerEU = 1;  // one problem per compute unit in any case
};
// The count window's rebuild takes rank r on thread r (wave w builds word w).
static_assert(LdsSmall::kT == LdsSmall::kTW * kWave && LdsTiny::kT == LdsTiny::kTW * kWave &&
                  LdsLarge::kT == LdsLarge::kTW * kWave,
              "one thread per rank of the largest R of each configuration");
// list entries pack (slot, slot-expert index, host structure): 12 + 7 + 7 bits
constexpr int kItemSlotBits = 12, kItemExpertBits = 7;

// Exclusive position of `flag` among the NT threads (ascending thread id) and
// the chunk total.  All threads must call it.
template <int NT>
__device__ __forceinline__ int32_t compact_pos_n(bool flag, int32_t* wave_cnt, int32_t& total) {
  constexpr int NW = NT / kWave;
  const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
  const uint64_t m = __ballot(flag);
  const int32_t lp = __popcll(m & ((1ull << lane) - 1ull));
  if (lane == 0) wave_cnt[wid] = __popcll(m);
  __syncthreads();
  int32_t off = 0, tot = 0;
  for (int w = 0; w < NW; ++w) {
    const int32_t c = wave_cnt[w];
    off += w < wid ? c : 0;
    tot += c;
  }
  __syncthreads();
  total = tot;
  return off + lp;
}

// Tier structure of column h of Bauct: its distinct bonuses in descending
// order and the rank set of each ([h][kTierMax][TW] words); ntier[h] = -1 if
// there are more than kTierMax.  NaN and -inf bonuses never win a bid and
// belong to no tier; -0 and +0 are one value.  The distinct values come out
// one per step as a block maximum over the values below the previous one
// (order-preserving 64-bit keys).
__device__ __forceinline__ double key_double(uint64_t k) {
  return __longlong_as_double((long long)((k >> 63) ? (k & 0x7FFFFFFFFFFFFFFFull) : ~k));
}

template <int NT>
__device__ __forceinline__ uint64_t block_max_u64(uint64_t v, uint64_t* buf) {
  constexpr int NW = NT / kWave;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t y = __shfl_xor(v, o, kWave);
    v = y > v ? y : v;
  }
  if ((threadIdx.x & (kWave - 1)) == 0) buf[threadIdx.x / kWave] = v;
  __syncthreads();
  uint64_t m = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) m = buf[w] > m ? buf[w] : m;
  __syncthreads();
  return m;
}

template <int TW>
__global__ void __launch_bounds__(256)
auction_tiers_kernel(const double* __restrict__ Bauct, int32_t R, int32_t* __restrict__ ntier,
                     double* __restrict__ tv, uint64_t* __restrict__ tmask) {
  __shared__ double col[TW * kWave];
  __shared__ double vals[kTierMax];
  __shared__ uint64_t red[256 / kWave];
  __shared__ unsigned long long msk[kTierMax * TW];
  const int32_t h = blockIdx.x, tid = threadIdx.x;
  for (int32_t q = tid; q < kTierMax * TW; q += blockDim.x) msk[q] = 0ull;
  for (int32_t r = tid; r < R; r += blockDim.x) col[r] = Bauct[(int64_t)r * R + h];
  __syncthreads();
  // the tier bonuses, descending: key 0 is below every value's key
  uint64_t prev = ~0ull;
  int32_t n = 0;
  for (int t = 0; t <= kTierMax; ++t) {
    uint64_t m = 0;
    for (int32_t r = tid; r < R; r += blockDim.x) {
      const double v = col[r];
      if (v != v || v == -INFINITY) continue;
      const uint64_t k = auction_key(v);
      if (k < prev && k > m) m = k;
    }
    m = block_max_u64<256>(m, red);
    if (m == 0) break;  // no value below the previous one
    if (t == kTierMax) { n = -1; break; }
    if (tid == 0) vals[t] = key_double(m);
    prev = m;
    n = t + 1;
  }
  __syncthreads();
  for (int32_t r = tid; r < R && n > 0; r += blockDim.x) {
    const double v = col[r];
    for (int32_t i = 0; i < n; ++i)
      if (vals[i] == v) atomicOr(&msk[i * TW + (r >> 6)], 1ull << (r & 63));
  }
  __syncthreads();
  if (tid == 0) ntier[h] = n;
  if (tid < kTierMax) tv[(int64_t)h * kTierMax + tid] = tid < n ? vals[tid] : -INFINITY;
  for (int32_t q = tid; q < kTierMax * TW; q += blockDim.x)
    tmask[(int64_t)h * kTierMax * TW + q] = q / TW < n ? msk[q] : 0ull;
}

// Deduplicates the host tier structures into a table of at most SC entries
// (one block, one thread per host; equal structures are found through a hash
// of each and then compared in full; the table keeps first occurrences in
// host order) and ranks the table's distinct bonuses (ascending, one per step
// as a block minimum above the previous one): sidx[h] is host h's entry, cw
// the words that hold ranks of each tier, cvr the bonus rank of each tier,
// hdr[0] the table size and hdr[1] = 1 when the LDS-resident auction is exact
// for this Bauct and price step: every column has at most kTierMax values,
// none is +inf, the table fits, and both the step (if not 0) and every gap
// between distinct bonuses exceed twice the spacing of doubles at max|bonus|
// + S * step (prices stay below S * step: a rank serves each slot at most
// once).
template <class CF>
__global__ void __launch_bounds__(CF::kT)
auction_struct_kernel(const int32_t* __restrict__ ntier_g, const double* __restrict__ tv_g,
                      const uint64_t* __restrict__ tmask, int32_t R, int64_t S, double step,
                      int32_t* __restrict__ sidx, int32_t* __restrict__ cn, double* __restrict__ cv,
                      int32_t* __restrict__ cvr, uint32_t* __restrict__ cw, uint64_t* __restrict__ cm,
                      int32_t* __restrict__ hdr) {
  constexpr int NT = CF::kT;
  constexpr int kRow = kTierMax * CF::kTW;
  constexpr int kMaxR = CF::kTW * kWave;
  constexpr int kMaxDv = CF::kSC * kTierMax;
  static_assert(NT >= kMaxR, "one thread per host");
  __shared__ int32_t ntier[kMaxR], first[kMaxR], sid[kMaxR], tab[CF::kSC];
  __shared__ uint64_t hsh[kMaxR];
  __shared__ double tv[kMaxR * kTierMax];
  __shared__ double dv[kMaxDv];
  __shared__ uint64_t red[NT / kWave];
  __shared__ int32_t wave_cnt[NT / kWave];
  const int32_t h = threadIdx.x;
  for (int32_t q = h; q < R * kTierMax; q += NT) tv[q] = tv_g[q];
  if (h < R) {
    const int32_t nh = ntier_g[h];
    ntier[h] = nh;
    uint64_t x = 0x9E3779B97F4A7C15ull ^ (uint64_t)(uint32_t)nh;
    for (int32_t t = 0; t < kTierMax; ++t) {
      x = (x ^ (uint64_t)__double_as_longlong(tv_g[h * kTierMax + t])) * 0x100000001B3ull;
      x ^= x >> 29;
    }
    for (int32_t q = 0; q < kRow; ++q) {
      x = (x ^ tmask[(int64_t)h * kRow + q]) * 0x100000001B3ull;
      x ^= x >> 29;
    }
    hsh[h] = x;
  }
  __syncthreads();
  if (h < R) {
    const int32_t nh = ntier[h];
    int32_t f = h;
    for (int32_t g = 0; g < h && f == h; ++g) {
      if (hsh[g] != hsh[h] || ntier[g] != nh) continue;
      bool eq = true;
      for (int32_t t = 0; t < kTierMax && eq; ++t) eq = tv[g * kTierMax + t] == tv[h * kTierMax + t];
      for (int32_t q = 0; q < kRow && eq; ++q) eq = tmask[(int64_t)g * kRow + q] == tmask[(int64_t)h * kRow + q];
      if (eq) f = g;
    }
    first[h] = f;
  }
  __syncthreads();
  // table entries: the first occurrences in host order
  int32_t ns;
  {
    const bool f = h < R && first[h] == h;
    const int32_t pos = compact_pos_n<NT>(f, wave_cnt, ns);
    if (f) {
      sid[h] = pos;
      if (pos < CF::kSC) tab[pos] = h;
    }
  }
  __syncthreads();
  if (h < R && first[h] != h) sid[h] = sid[first[h]];
  // exactness conditions over all hosts: at most kTierMax values per column,
  // no +inf, and max |bonus|
  bool okh = true;
  uint64_t vmk = 0;  // bits of max |bonus| (non-negative doubles order as integers)
  if (h < R) {
    okh = ntier[h] >= 0;
    for (int32_t t = 0; t < ntier[h]; ++t) {
      const double v = tv[h * kTierMax + t];
      okh &= v != INFINITY;
      const uint64_t a = (uint64_t)__double_as_longlong(fabs(v));
      vmk = a > vmk ? a : vmk;
    }
  }
  const bool all_ok = block_max_u64<NT>(okh ? 0ull : 1ull, red) == 0ull;
  const double vm = __longlong_as_double((long long)block_max_u64<NT>(vmk, red));
  // distinct bonuses of the table, ascending: value q is tier q % kTierMax of
  // entry q / kTierMax, dealt out over the threads
  const int32_t nt_tab = ns < CF::kSC ? ns : CF::kSC;
  int32_t nd = 0;
  {
    uint64_t prev = 0;  // keys above this; the smallest first
    for (;;) {
      // minimum key above prev, as a maximum of complements
      uint64_t c = 0;
      for (int32_t q = h; q < nt_tab * kTierMax; q += NT) {
        const int32_t g = tab[q / kTierMax], t = q % kTierMax;
        if (t >= ntier[g]) continue;
        const uint64_t k = auction_key(tv[g * kTierMax + t]);
        if (k > prev && ~k > c) c = ~k;
      }
      const uint64_t m = block_max_u64<NT>(c, red);
      if (m == 0) break;
      const uint64_t kmin = ~m;
      if (h == 0 && nd < kMaxDv) dv[nd] = key_double(kmin);
      prev = kmin;
      ++nd;
    }
  }
  __syncthreads();
  if (h == 0) {
    bool ok = all_ok && ns <= CF::kSC;
    const double top = vm + (double)S * step * 1.01 + 1.0;
    const double spacing2 = 2.0 * (nextafter(top, INFINITY) - top);
    ok &= step == 0.0 || (step > 0.0 && step > spacing2);
    for (int32_t i = 0; i + 1 < nd; ++i) ok &= dv[i + 1] - dv[i] > spacing2;
    hdr[0] = nt_tab;
    hdr[1] = ok ? 1 : 0;
  }
  // bonus ranks of the table's tiers
  for (int32_t q = h; q < nt_tab * kTierMax; q += NT) {
    const int32_t g = tab[q / kTierMax], t = q % kTierMax;
    int32_t rank = 0;
    if (t < ntier[g]) {
      const double v = tv[g * kTierMax + t];
      while (dv[rank] != v) ++rank;
    }
    cvr[q] = rank;
  }
  for (int32_t q = h; q < R; q += NT) sidx[q] = sid[q];
  for (int32_t q = h; q < nt_tab; q += NT) cn[q] = ntier[tab[q]] > 0 ? ntier[tab[q]] : 0;
  for (int32_t q = h; q < nt_tab * kTierMax; q += NT) {
    const int32_t g = tab[q / kTierMax], t = q % kTierMax;
    cv[q] = tv[g * kTierMax + t];
    uint32_t words = 0;
    for (int32_t w = 0; w < CF::kTW; ++w) words |= (tmask[(int64_t)g * kRow + t * CF::kTW + w] != 0ull ? 1u : 0u) << w;
    cw[q] = words;
  }
  for (int32_t q = h; q < nt_tab * kRow; q += NT) cm[q] = tmask[(int64_t)tab[q / kRow] * kRow + q % kRow];
}

template <class CF>
struct LdsState {
  // both phases
  int16_t* slot_ec;   // [S] candidate index of the slot's expert or -1
  int32_t* amt;       // [S] slot amounts (Phase 2), tokens still planned (Phase 3)
  int32_t* ce;        // [NEC] candidate experts (spill > 0), ascending
  // Phase 2
  int32_t* hce; double* den; int32_t* cr; int32_t* spare_p; int32_t* matched; int32_t* prop_e;
  double* prop_s; int32_t* assigned; int32_t* spill_p; uint64_t* ekey; int32_t* ewin;
  int32_t* qbest;  // [R] q = min(spill, spare) of each cold rank's standing proposal
  // Phase 3 (aliases the Phase-2 region)
  double* price; uint32_t* rkey; int32_t* work; uint16_t* sstate;
  uint64_t* vmask; uint32_t* vwords; int32_t* dexp; int32_t* dmap; int32_t* cnt; uint64_t* planes;
  // relative counts: lvl0 [TW] the ranks at the base count, lvl1 [TW] those
  // one service above it, rel [kRelPlanes] [TW] the code planes, p0 the
  // price of the base count; misc: base,
  // minimum (rebase scratch), a base-count word emptied (2, by round parity),
  // a transfer made (2, by round parity), the base's epoch (rebases so far)
  uint64_t* lvl0; uint64_t* lvl1; uint64_t* rel; double* p0; int32_t* misc;
  int8_t* cn; double* cv; int32_t* cvr; uint32_t* cw; uint64_t* cm;
  size_t bytes;
};

template <class CF>
__host__ __device__ inline LdsState<CF> carve_lds(char* base, int32_t R, int32_t K, int32_t NEC) {
  LdsState<CF> w;
  const size_t S1 = R * K > 0 ? (size_t)R * K : 1, R_ = (size_t)R, N_ = (size_t)NEC;
  constexpr size_t TW = CF::kTW, SC = CF::kSC, DC = CF::kDC;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* q = base + off;
    off = (off + bytes + 15) & ~(size_t)15;
    return q;
  };
  w.slot_ec = (int16_t*)take(2 * S1);
  w.amt = (int32_t*)take(4 * S1);
  w.ce = (int32_t*)take(4 * N_);
  const size_t split = off;
  w.hce = (int32_t*)take(4 * N_); w.den = (double*)take(8 * R_); w.cr = (int32_t*)take(4 * R_);
  w.spare_p = (int32_t*)take(4 * R_); w.matched = (int32_t*)take(4 * R_); w.prop_e = (int32_t*)take(4 * R_);
  w.prop_s = (double*)take(8 * R_); w.assigned = (int32_t*)take(4 * S1);
  w.spill_p = (int32_t*)take(4 * N_); w.ekey = (uint64_t*)take(8 * N_); w.ewin = (int32_t*)take(4 * N_);
  w.qbest = (int32_t*)take(4 * R_);
  const size_t end2 = off;
  off = split;
  w.price = (double*)take(8 * R_); w.rkey = (uint32_t*)take(4 * R_);
  w.work = (int32_t*)take(4 * S1);
  // bid states of the packed layout's list entries, by list position
  // (several waves, at most two slots per thread; the 4-wave build for few
  // problems per compute unit leaves them unused)
  w.sstate = (uint16_t*)take(CF::kT > kWave && S1 <= 2 * (size_t)CF::kT ? 2 * S1 : 0);
  // the word lists guide the per-word search of sets wider than 4 words only
  w.vmask = (uint64_t*)take(8 * DC * TW); w.vwords = (uint32_t*)take(TW > 4 ? 4 * DC : 0);
  w.dexp = (int32_t*)take(4 * DC); w.dmap = (int32_t*)take(4 * N_);
  w.cnt = (int32_t*)take(4 * R_); w.planes = (uint64_t*)take(8 * CF::kPL * TW);
  w.lvl0 = (uint64_t*)take(8 * TW); w.lvl1 = (uint64_t*)take(8 * TW);
  w.rel = (uint64_t*)take(8 * kRelPlanes * TW);
  w.p0 = (double*)take(8); w.misc = (int32_t*)take(4 * 8);
  w.cn = (int8_t*)take(SC);
  w.cv = (double*)take(8 * SC * kTierMax); w.cvr = (int32_t*)take(4 * SC * kTierMax);
  w.cw = (uint32_t*)take(4 * SC * kTierMax);
  w.cm = (uint64_t*)take(8 * SC * kTierMax * TW);
  w.bytes = end2 > off ? end2 : off;
  return w;
}

struct LdsParams {
  SchParams s;
  const int32_t* sidx;   // [R] host -> tier structure
  const int32_t* cn;     // [SC] tiers per structure
  const double* cv;      // [SC][kTierMax] tier bonuses, descending
  const int32_t* cvr;    // [SC][kTierMax] rank of each tier bonus among the table's
  const uint32_t* cw;    // [SC][kTierMax] words holding ranks of the tier
  const uint64_t* cm;    // [SC][kTierMax][TW] tier rank sets
  const int32_t* hdr;    // [0] structures, [1] LDS-resident auction exact
  int32_t* fallback;     // [B] 1 = left to schedule_kernel
  int32_t* nprime;       // [B][DC][R]
  int32_t NEC;           // candidate-expert capacity of the LDS layout
  int32_t shared;        // 1 when the batch has more problems than compute units
};

// Block-wide OR with one barrier; flags alternate between two halves of buf
// ([2][NT / 64]) so that a call never overwrites flags still being read.
template <int NT>
__device__ __forceinline__ bool block_or(bool flag, int32_t* buf, int& parity) {
  constexpr int NW = NT / kWave;
  const uint64_t m = __ballot(flag);
  if ((threadIdx.x & (kWave - 1)) == 0) buf[parity * NW + threadIdx.x / kWave] = m != 0;
  __syncthreads();
  bool any = false;
#pragma unroll
  for (int w = 0; w < NW; ++w) any |= buf[parity * NW + w] != 0;
  parity ^= 1;
  return any;
}

// Appends the flagged items of a wave to a list whose length lives in LDS
// (*count); the order of the list is unspecified.  All lanes must call it;
// a flagged lane gets its item's position.
__device__ __forceinline__ int32_t list_append(bool flag, int32_t item, int32_t* list, int32_t* count) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint64_t m = __ballot(flag);
  int32_t base = 0;
  if (lane == 0 && m) base = atomicAdd(count, __popcll(m));
  base = __builtin_amdgcn_readlane(base, 0);
  const int32_t pos = base + __popcll(m & ((1ull << lane) - 1ull));
  if (flag) list[pos] = item;
  return pos;
}

template <int CTRL>
__device__ __forceinline__ int32_t dpp_i32(int32_t x) {
  // every lane has a source lane for the patterns used here
  return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xf, 0xf, true);
}
// Max over the 64 lanes without LDS round trips: DPP steps within each
// 16-lane row, then the permlane16 and permlane32 swaps across rows.  All
// lanes must call it.
__device__ __forceinline__ int32_t wave_max_i32(int32_t v) {
  v = max(v, dpp_i32<0xB1>(v));   // quad_perm [1,0,3,2]
  v = max(v, dpp_i32<0x4E>(v));   // quad_perm [2,3,0,1]
  v = max(v, dpp_i32<0x141>(v));  // row_half_mirror
  v = max(v, dpp_i32<0x140>(v));  // row_mirror
  const auto r16 = __builtin_amdgcn_permlane16_swap((uint32_t)v, (uint32_t)v, false, false);
  v = max((int32_t)r16[0], (int32_t)r16[1]);
  const auto r32 = __builtin_amdgcn_permlane32_swap((uint32_t)v, (uint32_t)v, false, false);
  return max((int32_t)r32[0], (int32_t)r32[1]);
}

// One problem per workgroup of CF::kT threads; thread i bids for list entries
// i, i + kT, ... (SPL of them).  WPE waves per SIMD bound the registers: a
// batch that fills the chip needs all its problems resident at once, a
// smaller one is better served without the register cap.
template <class CF, int SPL, int WPE>
__global__ void __launch_bounds__(CF::kT, WPE) schedule_lds_kernel(LdsParams wp) {
  constexpr int NT = CF::kT, NW = NT / kWave, TW = CF::kTW;
  extern __shared__ __attribute__((aligned(16))) char lds_dyn[];
  __shared__ int32_t wave_cnt[NW];
  __shared__ int32_t flagbuf[2 * NW];
  __shared__ int32_t sh_maxc, sh_nw[2];
  __shared__ unsigned long long sh_sum, sh_big;
  const SchParams& p = wp.s;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
  const int64_t b = blockIdx.x;
  const int32_t R = p.R, E = p.E, K = p.K;
  const int32_t S = R * K;
  int parity = 0;
  LdsState<CF> L = carve_lds<CF>(lds_dyn, R, K, wp.NEC);

  if (wp.hdr[1] == 0) {  // the LDS-resident auction would not be exact for this Bauct and step
    if (tid == 0) wp.fallback[b] = 1;
    return;
  }
  const int64_t* spill = p.spill + b * E;
  const int64_t* spare = p.spare + b * R;
  const int64_t* excess = p.excess + b * R;
  const float* Tb = p.T + b * (int64_t)R * R;
  int32_t* se = p.slot_expert + b * S;
  int64_t* sa = p.slot_amount + b * S;
  int32_t* Xb = p.X + b * (int64_t)R * S;
  const double alpha = topo_weight(p.flags, p.alpha[b]);
  const double a2 = flow_weight(p.flags, p.alpha[b]);

  // ---- validation, candidates, cold ranks ------------------------------------------
  bool badh = false;
  for (int32_t e = tid; e < E; e += NT) {
    const int32_t h = p.home[e];
    badh |= h < 0 || h >= R;
  }
  if (tid == 0) { sh_sum = 0; sh_big = 0; sh_maxc = 0; }
  if (block_or<NT>(badh, flagbuf, parity)) {
    for (int32_t s = tid; s < S; s += NT) { se[s] = -1; sa[s] = 0; }
    for (int64_t q = tid; q < (int64_t)R * S; q += NT) Xb[q] = 0;
    if (tid == 0) {
      p.unfilled[b] = 0;
      if (p.rounds_used) { p.rounds_used[2 * b] = 0; p.rounds_used[2 * b + 1] = 0; }
      if (p.status) p.status[b] = TAOT_ST_BAD_INPUT;
      wp.fallback[b] = 0;
    }
    return;
  }
  int32_t ne = 0, nc = 0;
  int64_t mass = 0, big = 0;  // amounts must fit the 32-bit LDS state
  for (int32_t base = 0; base < E; base += NT) {
    const int32_t e = base + tid;
    const int64_t v = e < E ? spill[e] : 0;
    const bool f = v > 0;
    int32_t tot;
    const int32_t pos = ne + compact_pos_n<NT>(f, wave_cnt, tot);
    if (f && pos < wp.NEC) {
      L.ce[pos] = e;
      L.spill_p[pos] = (int32_t)(v < INT_MAX ? v : INT_MAX);
      L.hce[pos] = p.home[e];
    }
    ne += tot;
    mass += f ? v : 0;
  }
  for (int32_t base = 0; base < R; base += NT) {
    const int32_t r = base + tid;
    const int64_t v = r < R ? spare[r] : 0;
    const bool f = v > 0;
    int32_t tot;
    const int32_t pos = nc + compact_pos_n<NT>(f, wave_cnt, tot);
    if (f) { L.cr[pos] = r; L.spare_p[pos] = (int32_t)(v < INT_MAX ? v : INT_MAX); }
    nc += tot;
    big = v > big ? v : big;
    if (r < R) {
      const double ex = (double)excess[r];
      L.den[r] = ex > kEps0 ? ex : kEps0;
    }
  }
  mass = wave_sum_i64(mass);
  big = wave_max_i64(big);
  if (lane == 0) {
    atomicAdd(&sh_sum, (unsigned long long)mass);
    atomicMax(&sh_big, (unsigned long long)big);
  }
  __syncthreads();
  if (ne > wp.NEC || sh_sum > (unsigned long long)INT_MAX || sh_big > (unsigned long long)INT_MAX) {
    if (tid == 0) wp.fallback[b] = 1;
    return;
  }
  for (int32_t q = tid; q < nc * K; q += NT) L.assigned[q] = -1;
  for (int32_t ec = tid; ec < ne; ec += NT) { L.ekey[ec] = 0; L.ewin[ec] = INT_MAX; }
  for (int32_t s = tid; s < S; s += NT) { L.slot_ec[s] = -1; L.amt[s] = 0; se[s] = -1; }
  __syncthreads();

  // ---- Phase 2: column-priority iterative matching ---------------------------------
  int32_t used2 = 0;
  for (int32_t k = 0; k < K; ++k) {
    for (int32_t rc = tid; rc < nc; rc += NT) { L.matched[rc] = 0; L.prop_e[rc] = -1; }
    __syncthreads();
    for (int32_t inner = 0; inner < nc; ++inner) {
      // Step 1: every unmatched cold rank proposes its best candidate expert
      bool proposed = false;
      for (int32_t rc = tid; rc < nc; rc += NT) {
        if (L.matched[rc]) continue;
        const int32_t sp = L.spare_p[rc];
        // A losing proposal stands while its expert's q = min(spill, spare) is
        // unchanged: within a round of k no score rises (spill only falls; an
        // unmatched rank's spare, its taken set and the other terms are
        // fixed), so that expert is still the best, and still the lowest
        // index among the best.  Otherwise the rank scans again.
        const int32_t pe = L.prop_e[rc];
        if (pe >= 0) {
          const int32_t sl = L.spill_p[pe];
          if ((sl < sp ? sl : sp) == L.qbest[rc]) {
            proposed = true;
            continue;
          }
        }
        int32_t best = -1, bq = 0;
        double bs = -INFINITY;
        if (sp > 0) {
          const int32_t r = L.cr[rc];
          const int32_t* asg = L.assigned + rc * K;
          const int32_t a0 = k > 0 ? asg[0] : -1, a1 = k > 1 ? asg[1] : -1;
          const int32_t a2_ = k > 2 ? asg[2] : -1, a3 = k > 3 ? asg[3] : -1;
          for (int32_t ec0 = 0; ec0 < ne; ec0 += 4) {
            int32_t sl[4], hh[4];
            double bp[4];
            float tt[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const bool in = ec0 + u < ne;
              sl[u] = in ? L.spill_p[ec0 + u] : 0;
              hh[u] = in ? L.hce[ec0 + u] : r;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const bool ok = sl[u] > 0 && hh[u] != r;
              const int64_t o = (int64_t)hh[u] * R + r;
              bp[u] = ok ? p.Bpref[o] : 0.0;
              tt[u] = ok ? Tb[o] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int32_t ec = ec0 + u;
              if (sl[u] <= 0 || hh[u] == r) continue;
              bool taken = ec == a0 || ec == a1 || ec == a2_ || ec == a3;
              for (int32_t kk = 4; kk < k; ++kk) taken |= asg[kk] == ec;
              if (taken) continue;
              const double q = (double)(sl[u] < sp ? sl[u] : sp);
              const double t1 = alpha * bp[u];
              const double tn = (double)tt[u] / L.den[hh[u]];
              const double t2 = a2 * tn;
              const double score = (q + t1) + t2;
              if (score > bs) { bs = score; best = ec; bq = sl[u] < sp ? sl[u] : sp; }
            }
          }
        }
        L.prop_e[rc] = best;
        L.prop_s[rc] = bs;
        L.qbest[rc] = bq;
        proposed |= best >= 0;
      }
      if (!block_or<NT>(proposed, flagbuf, parity)) break;  // nothing can change any more
      // Steps 2-3: each proposed expert keeps its best proposer: max score, then lowest rank
      for (int32_t rc = tid; rc < nc; rc += NT)
        if (L.prop_e[rc] >= 0)
          atomicMax(reinterpret_cast<unsigned long long*>(&L.ekey[L.prop_e[rc]]),
                    (unsigned long long)ordered_key(L.prop_s[rc]));
      __syncthreads();
      for (int32_t rc = tid; rc < nc; rc += NT)
        if (L.prop_e[rc] >= 0 && ordered_key(L.prop_s[rc]) == L.ekey[L.prop_e[rc]])
          atomicMin(&L.ewin[L.prop_e[rc]], rc);
      __syncthreads();
      // Step 4: winners take g = min(spill, spare) into slot k of their rank
      for (int32_t ec = tid; ec < ne; ec += NT) {
        const int32_t w = L.ewin[ec];
        if (w != INT_MAX) {
          const int32_t g = L.spill_p[ec] < L.spare_p[w] ? L.spill_p[ec] : L.spare_p[w];
          L.spill_p[ec] -= g;
          L.spare_p[w] -= g;
          L.matched[w] = 1;
          L.prop_e[w] = -1;  // matched ranks stop proposing
          L.assigned[w * K + k] = ec;
          const int32_t s = L.cr[w] * K + k;
          L.slot_ec[s] = (int16_t)ec;
          L.amt[s] += g;
          se[s] = L.ce[ec];
        }
        L.ekey[ec] = 0;
        L.ewin[ec] = INT_MAX;
      }
      __syncthreads();
      ++used2;
    }
  }
  for (int32_t s = tid; s < S; s += NT) sa[s] = L.amt[s];

  // ---- Phase 3: Lagrangian auction ---------------------------------------------------
  // distinct slot experts, in ascending candidate (= expert) order
  __syncthreads();
  for (int32_t ec = tid; ec < ne; ec += NT) L.dmap[ec] = 0;
  __syncthreads();
  for (int32_t s = tid; s < S; s += NT)
    if (L.slot_ec[s] >= 0) L.dmap[L.slot_ec[s]] = 1;
  __syncthreads();
  int32_t D = 0;
  for (int32_t base = 0; base < ne; base += NT) {
    const int32_t ec = base + tid;
    const bool f = ec < ne && L.dmap[ec] == 1;
    int32_t tot;
    const int32_t pos = D + compact_pos_n<NT>(f, wave_cnt, tot);
    if (ec < ne) L.dmap[ec] = f ? pos : -1;
    if (f && pos < CF::kDC) L.dexp[pos] = L.ce[ec];
    D += tot;
  }
  if (D > CF::kDC) {
    if (tid == 0) wp.fallback[b] = 1;
    return;
  }
  __syncthreads();
  // tokens of each slot expert per rank (device memory), the valid-rank sets
  // and the words of each set that hold ranks
  int32_t* np = wp.nprime + b * (int64_t)CF::kDC * R;
  const int32_t* nb = p.n + b * (int64_t)R * E;
  if constexpr (TW > 4)
    for (int32_t d = tid; d < D; d += NT) L.vwords[d] = 0u;
  __syncthreads();
  // (wave w takes word w, rank r on its lane; the strided loads of eight
  // experts are issued before any is used)
  static_assert(TW == NW, "one rank word per wave");
  {
    const int32_t r = wid * kWave + lane;
    for (int32_t d0 = 0; d0 < D; d0 += 8) {
      int32_t v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = d0 + u < D && r < R ? nb[(int64_t)r * E + L.dexp[d0 + u]] : 0;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int32_t d = d0 + u;
        if (d >= D) break;
        if (r < R) np[(int64_t)d * R + r] = v[u];
        const uint64_t m = __ballot(v[u] > 0);
        if (lane == 0) {
          L.vmask[d * TW + wid] = m;
          if constexpr (TW > 4)
            if (m) atomicOr(&L.vwords[d], 1u << wid);
        }
      }
    }
  }
  // the active-slot list of the first round: every slot with tokens planned
  // (packed layout: the first slot of each bid group, see below)
  // (the packed list pays where the bid search competes for issue slots: the
  // 16-wave layout, and the 4-wave one when it runs many problems per
  // compute unit; with few problems per compute unit a round is a chain of
  // latencies, and compacting the list only lengthens it)
  constexpr bool kPack = SPL <= 2 && (TW > 4 || (NW > 1 && WPE > 1));
  if (tid < 2) sh_nw[tid] = 0;
  auto slot_item = [&](int32_t s, bool& f) {
    const int32_t ec = s < S ? L.slot_ec[s] : -1;
    f = ec >= 0 && L.amt[s] > 0;
    return f ? s | (L.dmap[ec] << kItemSlotBits) | (wp.sidx[s / K] << (kItemSlotBits + kItemExpertBits)) : 0;
  };
  // packed layout: the next open slot of each slot's bid group (-1: none),
  // over the slot experts, which nothing reads once the items are built
  int16_t* const gnext = L.slot_ec;
  if constexpr (kPack) {
    // Bid groups.  Two open slots with the same host tier structure and the
    // same expert (the item's bits above the slot) make the same bid: the
    // search reads only those and the shared state.  Their keys then differ
    // in the slot alone, so the lower slot wins wherever both bid, and a
    // slot of a group can only be served once every lower open slot of the
    // group is full.  A group without a valid rank is without one for all
    // its slots (validity depends on the expert only).  So each group bids
    // with its lowest open slot only; when that slot fills, the next open
    // slot of the group takes its place (and its bid state, which depends on
    // the group alone).  The rounds, bids and transfers are the same as
    // with every open slot bidding.  The items are built once, by slot, in
    // the list array (-1: no tokens planned).
    for (int32_t s = tid; s < S; s += NT) {
      bool f;
      const int32_t item = slot_item(s, f);
      L.work[s] = f ? item : -1;
    }
    __syncthreads();
    for (int32_t s = tid; s < S; s += NT) {
      const int32_t it0 = L.work[s];
      int32_t nx = -1;
      if (it0 >= 0) {
        // the group key; a slot without tokens (-1) has key -1
        const int32_t k = it0 >> kItemSlotBits;
        int32_t q = s + 1;
        for (; q < S && (q & 3); ++q)
          if ((L.work[q] >> kItemSlotBits) == k) { nx = q; break; }
        if (nx < 0) {
          // four items per 16-byte load (the list array is 16-byte aligned)
          for (; q + 3 < S; q += 4) {
            const int4 w4 = *reinterpret_cast<const int4*>(L.work + q);
            const bool x0 = (w4.x >> kItemSlotBits) == k, x1 = (w4.y >> kItemSlotBits) == k,
                       x2 = (w4.z >> kItemSlotBits) == k, x3 = (w4.w >> kItemSlotBits) == k;
            if (x0 || x1 || x2 || x3) {
              nx = x0 ? q : x1 ? q + 1 : x2 ? q + 2 : q + 3;
              break;
            }
          }
          if (nx < 0)
            for (; q < S; ++q)
              if ((L.work[q] >> kItemSlotBits) == k) { nx = q; break; }
        }
      }
      gnext[s] = (int16_t)nx;
    }
    __syncthreads();
    // a slot with a lower open slot in its group waits: its item is marked
    // negative (one writer per slot)
    for (int32_t s = tid; s < S; s += NT)
      if (gnext[s] >= 0) L.work[gnext[s]] |= (int32_t)0x80000000u;
    __syncthreads();
    // the groups' first slots, compacted into the list of round 1 (odd)
    int32_t mine[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) mine[i] = i * NT + tid < S ? L.work[i * NT + tid] : -1;
    __syncthreads();  // every item is read before the list overwrites the array
#pragma unroll
    for (int i = 0; i < 2; ++i) list_append(mine[i] >= 0, mine[i], L.work, &sh_nw[1]);
  } else {
    __syncthreads();
    for (int32_t base = 0; base < S; base += NT) {
      const int32_t s = base + tid;
      bool f;
      const int32_t item = slot_item(s, f);
      list_append(f, item, L.work, &sh_nw[1]);  // the list of round 1 (odd)
    }
  }
  for (int32_t r = tid; r < R; r += NT) {
    L.price[r] = 0.0;
    L.rkey[r] = 0;
    L.cnt[r] = 0;
  }
  for (int32_t q = tid; q < CF::kPL * TW; q += NT) L.planes[q] = 0ull;
  // every rank starts with 0 services: at the base count 0, code 0
  for (int32_t q = tid; q < TW; q += NT) {
    const int32_t lo = q * kWave;
    L.lvl0[q] = lo >= R ? 0ull : (R - lo >= kWave ? ~0ull : (1ull << (R - lo)) - 1ull);
    L.lvl1[q] = 0ull;
  }
  for (int32_t q = tid; q < kRelPlanes * TW; q += NT) L.rel[q] = 0ull;
  if (tid < 8) L.misc[tid] = tid == 1 ? INT_MAX : 0;
  if (tid == 0) L.p0[0] = 0.0;
  const int32_t ns = wp.hdr[0];
  for (int32_t q = tid; q < ns; q += NT) L.cn[q] = (int8_t)wp.cn[q];
  for (int32_t q = tid; q < ns * kTierMax; q += NT) {
    L.cv[q] = wp.cv[q];
    L.cvr[q] = wp.cvr[q];
    L.cw[q] = wp.cw[q];
  }
  for (int32_t q = tid; q < ns * kTierMax * TW; q += NT) L.cm[q] = wp.cm[q];
  // X starts at zero; every (rank, slot) pair is served at most once (after a
  // transfer either the rank holds no more tokens of the slot's expert or the
  // slot is full), so transfers below are plain stores
  {
    int4* x4 = reinterpret_cast<int4*>(Xb);
    const int64_t n4 = ((int64_t)R * S) / 4;
    if ((reinterpret_cast<uintptr_t>(Xb) & 15u) == 0) {
      for (int64_t q = tid; q < n4; q += NT) x4[q] = make_int4(0, 0, 0, 0);
      for (int64_t q = n4 * 4 + tid; q < (int64_t)R * S; q += NT) Xb[q] = 0;
    } else {
      for (int64_t q = tid; q < (int64_t)R * S; q += NT) Xb[q] = 0;
    }
  }
  __syncthreads();

  // Every bid names a rank, which then serves its best bidder with a positive
  // amount; so every open slot with a valid rank bids again in every round.
  // A slot drops out once it is full or finds no valid rank (validity only
  // ends).  The layout of 16-word rank sets (one problem per compute unit)
  // and the 4-wave layout in its build for many problems per compute unit
  // keep a list of the open slots, packed into the first waves each round,
  // so that few waves issue the bid searches (there the search competes for
  // issue slots), with each slot's bid state in LDS; the one-wave layout,
  // the 4-wave layout with few problems per compute unit (a round is then a
  // chain of latencies) and the largest slot counts keep each slot and its
  // state with the thread that took it from the first round's list.  A
  // round is two steps, one barrier each, with
  // the list counts in two buffers by round parity and the list and the rank
  // keys in one (every thread has read its entries before the barrier that
  // precedes the rewrite; each rank's winner clears its key, and a bidder
  // that reads the key after that sees 0, not its own key, and loses as it
  // should):
  //   X: each open slot bids and posts its key to the rank it bid for;
  //   Y: the same thread moves tokens if its slot won, and keeps the slot
  //      while it still plans tokens; a transfer marks the round, and a round
  //      without one (no bid) ends the auction.
  // Incremental bids.  A slot keeps, while the base count stays (an epoch),
  // the first tier ts that holds a valid rank for it and a resume rank pos
  // such that no valid rank of tier ts below pos is at the base count.  Both
  // hold in later rounds: validity only ends and counts only rise.  So tiers
  // before ts are empty, and the lowest base-count rank of tier ts at or
  // after pos, when there is one, is the tier's fewest-services rank (score
  // bonus - P0); the later tiers follow with the usual pruning.  Otherwise
  // the full search runs from tier ts.  The bid rank becomes the next pos.
  const double step = p.price_step;
  const bool track = step > 0.0;  // counts order the prices; with step 0 all prices stay 0
  const int64_t tmax = p.t_max > 0 ? p.t_max : (int64_t)S * (R + 1);
  constexpr uint32_t kSlotMask = (1u << kItemSlotBits) - 1u, kExpMask = (1u << kItemExpertBits) - 1u;
  // Slot state: resume rank (bits 0-10), first tier (11-12), then the
  // epoch.  The packed layout keeps it in LDS in 16 bits beside the slot's
  // list entry (same position, read together with it), with the epoch's
  // parity (bit 13) and a valid bit (14): a listed slot's state is rewritten
  // in every round it bids, and the base moves at most once per round, so a
  // state read back is from the current epoch or the one before; a slot
  // that takes over a group gets the state of the slot it replaces.
  constexpr int kPosBits = 11, kTsBits = 2;
  static_assert(TW * kWave < (1 << kPosBits) && kTierMax <= (1 << kTsBits), "slot state fields");
  // pack the open slots into the first waves each round (several waves, at
  // most two slots per thread: the LDS of four does not hold their states)
  int32_t item[SPL];
  uint32_t state[SPL];
#pragma unroll
  for (int i = 0; i < SPL; ++i) {
    item[i] = i * NT + tid < sh_nw[1] ? L.work[i * NT + tid] : -1;
    state[i] = 0xFFFFFFFFu;  // no epoch matches it
  }
  if constexpr (kPack) {
    for (int32_t s = tid; s < S; s += NT) L.sstate[s] = 0;  // not valid
    __syncthreads();  // the first round reads states other threads cleared
  }
  int64_t rounds = 0;
  for (int64_t t = 1; t <= tmax; ++t) {
    const int cur = (int)(t & 1), prv = cur ^ 1;
    uint32_t* rk = L.rkey;
    const int32_t maxc = sh_maxc;
    const int32_t nplanes = maxc > 0 ? 32 - __builtin_clz((uint32_t)maxc) : 0;
    const double P0 = L.p0[0];
    const uint32_t epoch = (uint32_t)L.misc[6];
    const int32_t nw = sh_nw[cur];
    // When problems share a compute unit (up to eight at R = 256), the
    // kernel ends with the last of them: the wave that holds a round's
    // list takes an issue priority that grows with the list, so that the
    // problems with more open slot groups (more work left) go first.  A
    // problem alone on its compute unit, and the one-wave layout of the
    // small batches, only pay for the extra instructions.
    if (NT > kWave && wp.shared && wid == 0) {
      if (nw >= 32) __builtin_amdgcn_s_setprio(3);
      else if (nw >= 16) __builtin_amdgcn_s_setprio(2);
      else if (nw >= 4) __builtin_amdgcn_s_setprio(1);
      else __builtin_amdgcn_s_setprio(0);
    }
    if (kPack && tid == 0) sh_nw[prv] = 0;
    // ---- X: bids --------------------------------------------------------------------------
    int32_t bid[SPL], held[SPL];
    uint32_t key[SPL];
#pragma unroll
    for (int i = 0; i < SPL; ++i) {
      bid[i] = -1;
      key[i] = 0;
      held[i] = 0;
      if constexpr (kPack) {
        // the entry and its state are read together (states travel with
        // the list entries); positions past the list are read and dropped
        const int32_t q = i * NT + tid, qc = q < S ? q : 0;
        const int32_t wq = L.work[qc];
        const uint32_t sq = L.sstate[qc];
        item[i] = q < nw ? wq : -1;
        state[i] = sq;
      }
      const int32_t it = item[i];
      if (it < 0) continue;
      const int32_t s = it & kSlotMask, d = (it >> kItemSlotBits) & kExpMask;
      const int32_t st = it >> (kItemSlotBits + kItemExpertBits);
      // argmax over ranks holding tokens of the slot's expert of
      // Bauct[r][host] - price[r], lowest rank on ties, by tiers
      const int32_t nt = L.cn[st];
      const uint64_t* vm = L.vmask + d * TW;
      int32_t ts = 0, pos = 0;
      const bool st_ok = kPack ? ((state[i] >> 14) & 1u) && ((state[i] >> 13) & 1u) == (epoch & 1u)
                               : (state[i] >> (kPosBits + kTsBits)) == epoch;
      if (st_ok) {
        ts = (int32_t)((state[i] >> kPosBits) & ((1u << kTsBits) - 1u));
        pos = (int32_t)(state[i] & ((1u << kPosBits) - 1u));
      }
      double bs = -INFINITY;
      int32_t br = INT_MAX, bv = 0;
      int32_t nts = -1, npos = R;  // the new state: first tier with a valid rank, its base-count rank
      if constexpr (TW <= 4) {
        // rank sets of at most 4 words live in registers; the tier data is
        // read per tier (the registers of the capped builds are scarce)
        uint64_t valid[TW];
#pragma unroll
        for (int w = 0; w < TW; ++w) valid[w] = vm[w];
        // lowest valid rank of tier ti at the base count, at or after rank from
        auto scan0 = [&](int32_t ti, int32_t from) {
          const uint64_t* tm = L.cm + (st * kTierMax + ti) * TW;
          int32_t hit = INT_MAX;
#pragma unroll
          for (int w = TW - 1; w >= 0; --w) {
            uint64_t h = tm[w] & valid[w] & L.lvl0[w];
            h = w < (from >> 6) ? 0ull : w == (from >> 6) ? h & (~0ull << (from & 63)) : h;
            if (h) hit = w * kWave + __builtin_ctzll(h);
          }
          return hit;
        };
        // fewest services among the valid ranks of tier ti: the smallest
        // relative code, then (all saturated) the smallest count; one plane
        // per step; INT_MAX when the tier holds no valid rank
        auto deep = [&](int32_t ti) {
          const uint64_t* tm = L.cm + (st * kTierMax + ti) * TW;
          uint64_t c[TW], m[TW];
          uint64_t anyc = 0;
#pragma unroll
          for (int w = 0; w < TW; ++w) { c[w] = tm[w] & valid[w]; anyc |= c[w]; }
          if (!anyc) return (int32_t)INT_MAX;
          // no candidate is at the base count, so the lowest one a service
          // above it, when there is one, has the fewest services
          {
            int32_t r1 = INT_MAX;
#pragma unroll
            for (int w = TW - 1; w >= 0; --w) {
              const uint64_t h1 = c[w] & L.lvl1[w];
              if (h1) r1 = w * kWave + __builtin_ctzll(h1);
            }
            if (r1 != INT_MAX) return r1;
          }
          bool sat = true;
#pragma unroll 1
          for (int j = kRelPlanes - 1; j >= 0; --j) {
            uint64_t mm = 0;
#pragma unroll
            for (int w = 0; w < TW; ++w) { m[w] = c[w] & ~L.rel[j * TW + w]; mm |= m[w]; }
            sat &= mm == 0ull;
            if (mm) {
#pragma unroll
              for (int w = 0; w < TW; ++w) c[w] = m[w];
            }
          }
          if (sat && track) {
            for (int32_t j = nplanes - 1; j >= 0; --j) {
              uint64_t mm = 0;
#pragma unroll
              for (int w = 0; w < TW; ++w) { m[w] = c[w] & ~L.planes[j * TW + w]; mm |= m[w]; }
              if (mm) {
#pragma unroll
                for (int w = 0; w < TW; ++w) c[w] = m[w];
              }
            }
          }
          int32_t rr = INT_MAX;
#pragma unroll
          for (int w = TW - 1; w >= 0; --w)
            if (c[w]) rr = w * kWave + __builtin_ctzll(c[w]);
          return rr;
        };
        int32_t t0 = ts;
        bool resume_fail = false;  // tier ts holds no valid rank at the base count
        if (ts < nt) {
          const int32_t h = scan0(ts, pos);
          if (h != INT_MAX) {
            bs = L.cv[st * kTierMax + ts] - P0;
            br = h;
            bv = L.cvr[st * kTierMax + ts];
            nts = ts;
            npos = h;
            t0 = ts + 1;
          } else {
            resume_fail = true;
          }
        }
        for (int32_t ti = t0; ti < nt; ++ti) {
          const double v = L.cv[st * kTierMax + ti];
          if (v - P0 < bs) break;  // no score in this tier or the next reaches bs
          const int32_t h = resume_fail && ti == ts ? INT_MAX : scan0(ti, 0);
          const bool at0 = h != INT_MAX;  // a candidate at the base count: its price is P0
          const int32_t rr = at0 ? h : deep(ti);
          if (rr == INT_MAX) continue;  // no valid rank in this tier
          if (nts < 0) { nts = ti; npos = at0 ? h : R; }
          const double sc = v - (at0 ? P0 : L.price[rr]);
          if (sc > bs || (sc == bs && rr < br)) { bs = sc; br = rr; bv = L.cvr[st * kTierMax + ti]; }
        }
      } else {
        const uint32_t vw = L.vwords[d];
        // the structure's tier bonuses, bonus ranks and words, loaded once
        // (16-byte loads); the tier loop is unrolled so that they stay in
        // registers
        double cvv[kTierMax];
        int32_t cvrr[kTierMax];
        uint32_t cww[kTierMax];
        {
          const double2* cv2 = reinterpret_cast<const double2*>(L.cv + st * kTierMax);
          const double2 a = cv2[0], b2 = cv2[1];
          cvv[0] = a.x; cvv[1] = a.y; cvv[2] = b2.x; cvv[3] = b2.y;
          const int4 r4 = *reinterpret_cast<const int4*>(L.cvr + st * kTierMax);
          cvrr[0] = r4.x; cvrr[1] = r4.y; cvrr[2] = r4.z; cvrr[3] = r4.w;
          const uint4 w4 = *reinterpret_cast<const uint4*>(L.cw + st * kTierMax);
          cww[0] = w4.x; cww[1] = w4.y; cww[2] = w4.z; cww[3] = w4.w;
        }
        // lowest valid rank of a tier at the base count, at or after rank
        // from: the tier's words with valid ranks, ascending, one per step
        auto scan0 = [&](const uint64_t* tm, uint32_t words, int32_t from) {
          const int32_t wf = from >> 6;
          for (uint32_t ws = wf < 32 ? words & (~0u << wf) : 0u; ws; ws &= ws - 1u) {
            const int w = __builtin_ctz(ws);
            uint64_t h = tm[w] & vm[w] & L.lvl0[w];
            if (w == wf) h &= ~0ull << (from & 63);
            if (h) return w * kWave + __builtin_ctzll(h);
          }
          return (int32_t)INT_MAX;
        };
        // fewest services among the valid ranks of a tier: the smallest
        // relative code over its words with valid ranks, up to four words per
        // group (a bit-sliced minimum within the group; a group replaces the
        // best only with a smaller code, so equal codes keep the lower
        // words), then (all saturated) the bit-plane search over the full
        // counts; INT_MAX when the tier holds no valid rank
        auto deep = [&](const uint64_t* tm, uint32_t words) {
          int32_t rr = INT_MAX;
          uint32_t best = kRelMax + 1, cand = 0;
          for (uint32_t wl = words; wl;) {
            int wi[4];
            uint64_t c[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              wi[u] = wl ? __builtin_ctz(wl) : -1;
              wl &= wl - 1u;
            }
            uint64_t pl[kRelPlanes][4], l1[4];
            uint64_t any = 0;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int w = wi[u] < 0 ? 0 : wi[u];
              c[u] = wi[u] < 0 ? 0ull : tm[w] & vm[w];
              any |= c[u];
              cand |= (c[u] != 0ull ? 1u : 0u) << w;
              l1[u] = L.lvl1[w];
#pragma unroll
              for (int j = 0; j < kRelPlanes; ++j) pl[j][u] = L.rel[j * TW + w];
            }
            if (!any) continue;
            // no candidate is at the base count, so a candidate one service
            // above it has the fewest services: the first group (words
            // ascending) that holds one gives the lowest such rank
            {
              int32_t r1 = INT_MAX;
#pragma unroll
              for (int u = 3; u >= 0; --u) {
                const uint64_t h1 = c[u] & l1[u];
                if (h1) r1 = wi[u] * kWave + __builtin_ctzll(h1);
              }
              if (r1 != INT_MAX) return r1;
            }
            uint32_t code = 0;
#pragma unroll
            for (int j = kRelPlanes - 1; j >= 0; --j) {
              uint64_t m[4], mm = 0;
#pragma unroll
              for (int u = 0; u < 4; ++u) { m[u] = c[u] & ~pl[j][u]; mm |= m[u]; }
              if (mm) {
#pragma unroll
                for (int u = 0; u < 4; ++u) c[u] = m[u];
              } else {
                code |= 1u << j;
              }
            }
            if (code < best) {
              best = code;
#pragma unroll
              for (int u = 3; u >= 0; --u)
                if (c[u]) rr = wi[u] * kWave + __builtin_ctzll(c[u]);
            }
          }
          if (best == kRelMax && track) {
            // a word's minimum count is the planes where no candidate remained
            rr = INT_MAX;
            uint32_t cmin = 0xFFFFFFFFu;
            for (uint32_t ws = cand; ws; ws &= ws - 1) {
              const int w = __builtin_ctz(ws);
              uint64_t x = tm[w] & vm[w];
              uint32_t mn = 0;
              for (int32_t j = nplanes - 1; j >= 0; --j) {
                const uint64_t m = x & ~L.planes[j * TW + w];
                if (m) x = m;
                else mn |= 1u << j;
              }
              if (mn < cmin) {  // words ascend: equal counts keep the lower rank
                cmin = mn;
                rr = w * kWave + __builtin_ctzll(x);
              }
            }
          }
          return rr;
        };
        bool resume_fail = false;  // tier ts holds no valid rank at the base count
        int32_t t0 = ts;
        if (ts < nt) {
          // the register arrays indexed by ts without dynamic indexing
          const uint32_t cw_ts = ts == 0 ? cww[0] : ts == 1 ? cww[1] : ts == 2 ? cww[2] : cww[3];
          const int32_t h = scan0(L.cm + (st * kTierMax + ts) * TW, cw_ts & vw, pos);
          if (h != INT_MAX) {
            bs = (ts == 0 ? cvv[0] : ts == 1 ? cvv[1] : ts == 2 ? cvv[2] : cvv[3]) - P0;
            br = h;
            bv = ts == 0 ? cvrr[0] : ts == 1 ? cvrr[1] : ts == 2 ? cvrr[2] : cvrr[3];
            nts = ts;
            npos = h;
            t0 = ts + 1;
          } else {
            resume_fail = true;
          }
        }
#pragma unroll
        for (int ti = 0; ti < kTierMax; ++ti) {
          if (ti < t0) continue;
          if (ti >= nt) break;
          const double v = cvv[ti];
          if (v - P0 < bs) break;  // no score in this tier or the next reaches bs
          const uint32_t cwt = cww[ti] & vw;
          if (!cwt) continue;  // no valid rank in this tier
          const uint64_t* tm = L.cm + (st * kTierMax + ti) * TW;
          const int32_t h = resume_fail && ti == ts ? INT_MAX : scan0(tm, cwt, 0);
          const bool at0 = h != INT_MAX;  // a candidate at the base count: its price is P0
          const int32_t rr = at0 ? h : deep(tm, cwt);
          if (rr == INT_MAX) continue;  // no valid rank in this tier
          if (nts < 0) { nts = ti; npos = at0 ? h : R; }
          const double sc = v - (at0 ? P0 : L.price[rr]);
          if (sc > bs || (sc == bs && rr < br)) { bs = sc; br = rr; bv = cvrr[ti]; }
        }
      }
      if (nts >= 0) {
        if constexpr (kPack) {
          state[i] = (uint32_t)npos | ((uint32_t)nts << kPosBits) | ((epoch & 1u) << 13) | (1u << 14);
        } else {
          state[i] = (uint32_t)npos | ((uint32_t)nts << kPosBits) | (epoch << (kPosBits + kTsBits));
        }
      }
      if (br != INT_MAX) {
        bid[i] = br;
        key[i] = ((uint32_t)bv << 16) | (uint32_t)(0xFFFF - s);  // bonus, then lowest slot
        held[i] = np[(int64_t)d * R + br];
        atomicMax(&rk[br], key[i]);
      }
    }
    // the barrier orders the keys (LDS); the token loads above complete on
    // their own before Y uses them
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
    // ---- Y: transfers -----------------------------------------------------------------------
    // the flags of the next round (read by every thread before the barrier above)
    if (tid == 0) { L.misc[2 + prv] = 0; L.misc[4 + prv] = 0; }
#pragma unroll
    for (int i = 0; i < SPL; ++i) {
      const int32_t r = bid[i];
      // a slot without a bid has no valid rank left (validity only ends)
      bool keep = r >= 0;
      int32_t succ = -1;  // packed layout: the slot that takes over a filled slot's group
      if (keep && rk[r] == key[i]) {
        const int32_t s = item[i] & kSlotMask, d = (item[i] >> kItemSlotBits) & kExpMask;
        // the winner's reads first, so that they share one LDS round trip
        // (the stores below may alias them as far as the compiler knows)
        int32_t a = L.amt[s];
        const double pr = L.price[r];
        const int32_t c0 = L.cnt[r], base = L.misc[0];
        const int32_t gn = kPack ? (int32_t)gnext[s] : -1;
        rk[r] = 0u;  // the rank's key is cleared for the next round
        const uint64_t bit = 1ull << (r & 63);
        // A winner always moves tokens (x > 0): its rank held tokens of the
        // slot's expert when the slot bid (a valid rank), one slot at most is
        // served per rank and round, and a listed slot still plans tokens.  So
        // the price and count updates come first, while the token count loaded
        // with the bid (device memory) is still on its way.
        L.misc[4 + cur] = 1;
        L.price[r] = pr + step;
        if (track) {
          const int32_t c1 = c0 + 1;
          L.cnt[r] = c1;
          if (c1 > maxc) atomicMax(&sh_maxc, c1);  // a new largest count (rare)
          for (uint32_t flip = (uint32_t)(c0 ^ c1); flip; flip &= flip - 1)
            atomicXor(reinterpret_cast<unsigned long long*>(&L.planes[__builtin_ctz(flip) * TW + (r >> 6)]), bit);
          // the relative code rises by one (below saturation); a word of the
          // base-count set that empties is flagged for the round's end
          const int32_t k0 = c0 - base;
          if (k0 < kRelMax)
            for (uint32_t flip = (uint32_t)(k0 ^ (k0 + 1)); flip; flip &= flip - 1)
              atomicXor(reinterpret_cast<unsigned long long*>(&L.rel[__builtin_ctz(flip) * TW + (r >> 6)]), bit);
          if (k0 == 0) {
            const uint64_t old = atomicXor(reinterpret_cast<unsigned long long*>(&L.lvl0[r >> 6]), bit);
            if (old == bit) L.misc[2 + cur] = 1;
          }
          // the rank enters (code 0 -> 1) or leaves (1 -> 2) the set one above the base
          if (k0 == 0 || k0 == 1) atomicXor(reinterpret_cast<unsigned long long*>(&L.lvl1[r >> 6]), bit);
        }
        const int32_t have = held[i];
        const int32_t x = have < a ? have : a;
        Xb[(int64_t)r * S + s] = x;
        np[(int64_t)d * R + r] = have - x;
        a -= x;
        L.amt[s] = a;
        keep = a > 0;
        if (!keep) succ = gn;
        if (have - x <= 0) {
          const uint64_t old = atomicAnd(reinterpret_cast<unsigned long long*>(&L.vmask[d * TW + (r >> 6)]), ~bit);
          if constexpr (TW > 4)  // the word list only guides the per-word search
            if ((old & ~bit) == 0ull) atomicAnd(&L.vwords[d], ~(1u << (r >> 6)));
        }
      }
      if constexpr (kPack) {
        int32_t next = item[i];
        if (succ >= 0) {  // takes the filled slot's place and its bid state
          next = (next & ~(int32_t)kSlotMask) | succ;
          keep = true;
        }
        const uint16_t nst = (uint16_t)state[i];
        if (nw <= kWave) {
          // the round's whole list sits on wave 0 (entries 0 .. nw-1), so the
          // next one is compacted there without an atomic
          if (i == 0 && wid == 0) {
            const uint64_t m = __ballot(keep);
            if (keep) {
              const int32_t pos = (int32_t)__popcll(m & ((1ull << lane) - 1ull));
              L.work[pos] = next;
              L.sstate[pos] = nst;
            }
            if (lane == 0) sh_nw[prv] = (int32_t)__popcll(m);
          }
        } else {
          const int32_t pos = list_append(keep, next, L.work, &sh_nw[prv]);
          if (keep) L.sstate[pos] = nst;
        }
      } else if (!keep) {
        item[i] = -1;
      }
    }
    __syncthreads();
    if (!L.misc[4 + cur]) break;  // no bid this round: the state is final
    rounds = t;
    bool l0_empty = false;
    if (track && L.misc[2 + cur]) {
      l0_empty = true;
#pragma unroll
      for (int w = 0; w < TW; ++w) l0_empty &= L.lvl0[w] == 0ull;
    }
    if (l0_empty) {
      // Every rank has left the base count: the base moves to the new fewest
      // services and the relative codes are rebuilt from the counts.  Rank r
      // is thread r, so wave w builds word w; p0 takes the price of a rank at
      // the new base (every such rank has the same price).
      const int32_t mine = tid < R ? L.cnt[tid] : INT_MAX;
      const int32_t wmin = -wave_max_i32(-mine);
      if (lane == 0) atomicMin(&L.misc[1], wmin);
      __syncthreads();
      const int32_t nb = L.misc[1];
      const int32_t kr = tid < R ? min(L.cnt[tid] - nb, kRelMax) : -1;
      const uint64_t m0 = __ballot(kr == 0), m1 = __ballot(kr == 1);
      if (lane == 0 && wid < TW) {
        L.lvl0[wid] = m0;
        L.lvl1[wid] = m1;
      }
#pragma unroll
      for (int j = 0; j < kRelPlanes; ++j) {
        const uint64_t m = __ballot(kr > 0 && ((kr >> j) & 1));
        if (lane == 0 && wid < TW) L.rel[j * TW + wid] = m;
      }
      if (kr == 0) L.p0[0] = L.price[tid];
      __syncthreads();
      if (tid == 0) { L.misc[0] = nb; L.misc[1] = INT_MAX; L.misc[6] += 1; }
      __syncthreads();
    }
  }

  int64_t left = 0;
  // (a slot without an expert plans 0 tokens; the slot experts may hold the
  // bid groups' links by now)
  for (int32_t s = tid; s < S; s += NT) left += L.amt[s];
  left = wave_sum_i64(left);
  __syncthreads();
  if (tid == 0) sh_sum = 0;
  __syncthreads();
  if (lane == 0) atomicAdd(&sh_sum, (unsigned long long)left);
  __syncthreads();
  if (tid == 0) {
    const int64_t tot = (int64_t)sh_sum;
    p.unfilled[b] = tot;
    if (p.rounds_used) { p.rounds_used[2 * b] = used2; p.rounds_used[2 * b + 1] = (int32_t)rounds; }
    if (p.status) p.status[b] = tot > 0 ? TAOT_ST_UNFILLED : 0u;
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
  uint64_t* tmask;     // [R][kTierMax][TW]
  int32_t* sidx;       // [R]
  int32_t* cn;         // [SC]
  double* cv;          // [SC][kTierMax]
  int32_t* cvr;        // [SC][kTierMax]
  uint32_t* cw;        // [SC][kTierMax]
  uint64_t* cm;        // [SC][kTierMax][TW]
  int32_t* hdr;        // [2]
  int32_t* nprime;     // [B][DC][R]
  int64_t slab_bytes;
  size_t bytes;
};

// The tables are sized for the largest configuration, which any of them may use.
SchWs carve_sched(void* ws, int32_t B, int32_t R, int32_t E, int32_t K) {
  Carver c{static_cast<char*>(ws)};
  SchWs w;
  const bool lds_path = R <= LdsLarge::kTW * kWave;
  const size_t TW = LdsLarge::kTW, SC = LdsLarge::kSC, DC = lds_path ? LdsLarge::kDC : 0;
  w.slab_bytes = round_up((int64_t)carve_slab(nullptr, R, E, K).bytes, 256);
  w.slab = c.take<char>((size_t)w.slab_bytes * (B > 0 ? sched_grid(B) : 0));
  w.fallback = c.take<int32_t>((size_t)B);
  w.ntier = c.take<int32_t>((size_t)R);
  w.tv = c.take<double>((size_t)R * kTierMax);
  w.tmask = c.take<uint64_t>((size_t)R * kTierMax * TW);
  w.sidx = c.take<int32_t>((size_t)R);
  w.cn = c.take<int32_t>(SC);
  w.cv = c.take<double>(SC * kTierMax);
  w.cvr = c.take<int32_t>(SC * kTierMax);
  w.cw = c.take<uint32_t>(SC * kTierMax);
  w.cm = c.take<uint64_t>(SC * kTierMax * TW);
  w.hdr = c.take<int32_t>(2);
  w.nprime = c.take<int32_t>((size_t)B * DC * R);
  w.bytes = c.off;
  return w;
}

template <class CF, int SPL, int WPE>
taot_status launch_lds_kernel(const LdsParams& wp, int32_t B, size_t lds, hipStream_t stream) {
  if (lds > 65536 && hipFuncSetAttribute((const void*)schedule_lds_kernel<CF, SPL, WPE>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return TAOT_ERR_LAUNCH;
  hipLaunchKernelGGL((schedule_lds_kernel<CF, SPL, WPE>), dim3((unsigned)B), dim3(CF::kT), lds, stream, wp);
  return hipGetLastError() == hipSuccess ? TAOT_OK : TAOT_ERR_LAUNCH;
}

// Largest dynamic LDS a workgroup may use on the current device.
size_t max_lds_per_block() {
  static size_t cached[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 65536;
  if (cached[dev] == 0) {
    int v = 0;
    cached[dev] = hipDeviceGetAttribute(&v, hipDeviceAttributeSharedMemPerBlockOptin, dev) == hipSuccess && v > 0
                      ? (size_t)v
                      : 65536;
  }
  return cached[dev];
}

// Prepasses and the LDS-resident kernel of configuration CF; false when its
// layout does not fit (the general kernel then takes every problem).
template <class CF>
taot_status launch_lds_path(const SchParams& p, const SchWs& w, int32_t B, int32_t R, int32_t E, int32_t K,
                            double price_step, hipStream_t stream, bool& launched) {
  launched = false;
  const int32_t NEC = E < CF::kNEC ? E : CF::kNEC;  // candidate experts (spill > 0) held in LDS
  const int64_t S = (int64_t)R * K;
  const size_t slds = carve_lds<CF>(nullptr, R, K, NEC).bytes;
  if (R > CF::kTW * kWave || S <= 0 || S > CF::kMaxS || slds > max_lds_per_block()) return TAOT_OK;
  hipLaunchKernelGGL(auction_tiers_kernel<CF::kTW>, dim3((unsigned)R), dim3(256), 0, stream, p.Bauct, R, w.ntier,
                     w.tv, w.tmask);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  hipLaunchKernelGGL(auction_struct_kernel<CF>, dim3(1), dim3(CF::kT), 0, stream, w.ntier, w.tv, w.tmask, R, S,
                     price_step, w.sidx, w.cn, w.cv, w.cvr, w.cw, w.cm, w.hdr);
  if (hipGetLastError() != hipSuccess) return TAOT_ERR_LAUNCH;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return TAOT_ERR_LAUNCH;
  const LdsParams wp{p, w.sidx, w.cn, w.cv, w.cvr, w.cw, w.cm, w.hdr, w.fallback, w.nprime, NEC, B > cus ? 1 : 0};
  taot_status st;
  // a batch of more problems than fit six to a compute unit takes the
  // register-capped build, which can hold CF::kWavesPerEU per SIMD
  const bool cap = (int64_t)B > (int64_t)6 * cus;
  if (S <= CF::kT)
    st = cap ? launch_lds_kernel<CF, 1, CF::kWavesPerEU>(wp, B, slds, stream)
             : launch_lds_kernel<CF, 1, 1>(wp, B, slds, stream);
  else if (S <= 2 * CF::kT)
    st = cap ? launch_lds_kernel<CF, 2, CF::kWavesPerEU>(wp, B, slds, stream)
             : launch_lds_kernel<CF, 2, 1>(wp, B, slds, stream);
  else
    st = cap ? launch_lds_kernel<CF, 4, CF::kWavesPerEU>(wp, B, slds, stream)
             : launch_lds_kernel<CF, 4, 1>(wp, B, slds, stream);
  launched = st == TAOT_OK;
  return st;
}

}  // namespace

size_t schedule_ws(int32_t B, int32_t R, int32_t E, int32_t K) { return carve_sched(nullptr, B, R, E, K).bytes; }

taot_status launch_schedule(const int32_t* n, const int64_t* spill, const int64_t* spare,
                            const int64_t* excess, const double* alpha, const int32_t* home,
                            const float* T, const double* Bpref, const double* Bauct, int32_t B,
                            int32_t R, int32_t E, int32_t K, double price_step, int64_t t_max,
                            uint32_t flags, int32_t* slot_expert, int64_t* slot_amount, int32_t* X,
                            int64_t* unfilled, int32_t* rounds_used, uint32_t* status, void* ws,
                            hipStream_t stream) {
  if (B == 0) return TAOT_OK;
  SchWs w = carve_sched(ws, B, R, E, K);
  SchParams p{n, spill, spare, excess, alpha, home, T, Bpref, Bauct, B, R, E, K, price_step, t_max,
              slot_expert, slot_amount, X, unfilled, rounds_used, status, w.slab, w.slab_bytes, w.fallback,
              flags};
  bool launched = false;
  taot_status st = TAOT_OK;
  // the row-priority ablation lives in the general kernel only
  if (!(flags & TAOT_SCH_ROW_PRIORITY)) {
    st = launch_lds_path<LdsTiny>(p, w, B, R, E, K, price_step, stream, launched);
    if (st == TAOT_OK && !launched) st = launch_lds_path<LdsSmall>(p, w, B, R, E, K, price_step, stream, launched);
    if (st == TAOT_OK && !launched) st = launch_lds_path<LdsLarge>(p, w, B, R, E, K, price_step, stream, launched);
  }
  if (st != TAOT_OK) return st;
  if (!launched) p.fallback = nullptr;  // the general kernel takes every problem
  const size_t lds = (size_t)R * (sizeof(double) + sizeof(uint64_t) + 2 * sizeof(int32_t));
  if (lds > 65536 && hipFuncSetAttribute((const void*)schedule_kernel,
                                         hipFuncAttributeMaxDynamicSharedMemorySize,
                                         (int)lds) != hipSuccess)
    return TAOT_ERR_LAUNCH;
  hipLaunchKernelGGL(schedule_kernel, dim3((unsigned)sched_grid(B)), dim3(kSchThreads), lds, stream, p);
  return hipGetLastError() == hipSuccess ? TAOT_OK : TAOT_ERR_LAUNCH;
}

}  // namespace taot
