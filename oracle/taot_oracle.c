/* Reference oracle for the TAOT per-step replica planner (see taot_oracle.h).
 *
 * TEST INFRASTRUCTURE ONLY: plain double-precision loops written from the
 * paper's definitions (Sec. 3 and Appendix A of "TAOT: Topology-Aware Optimal
 * Transport for Dynamic Expert Replica Placement in MoE Training").  Built
 * with -ffp-contract=off so every floating-point operation rounds on its own.
 *
 * Readings where the paper is silent or ambiguous (each is listed in the
 * design notes of the repository):
 *   - integer quantities (excess, spare, spill) use the integer mean
 *     m = floor(L / R); rho and alpha use the exact mean L / R;
 *   - Sinkhorn starts from g = 0 on all R columns (v = 1) and one iteration is
 *     a row (u) update followed by a column (v) update; the column cap is
 *     applied once, after the last iteration; eps0 = 1e-12;
 *   - every argmax is masked (non-candidates never win) and breaks ties
 *     towards the lowest index;
 *   - Phase-2 slots are s = r*K + k over all R ranks; Phase 3 stops after the
 *     first round without a bid, which leaves the state unchanged and is thus
 *     equivalent to running all t_max rounds;
 *   - topology preference B = cmin / C off the diagonal, 0 (Phase 2) or
 *     1 (Phase 3) on it.
 *
 * Parity unpinned: the Phase-2 and Phase-3 schedules have no worked example
 * in the paper, so their exact output is pinned only by invariants, the
 * relaxed-LP upper bound on tiny cases and hand-traced micro-cases.
 */
#include <omp.h>
#include "taot_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Loads (Sec. 3.1, Sec. A.1) and spill (Sec. A.3, cumulative-excess
 * differencing). */

static void plan_loads_one(const int32_t* ids, int32_t R, int64_t N, int32_t E, const int32_t* home,
                           int32_t* n, int64_t* x, int64_t* load, int64_t* excess, int64_t* spare,
                           int64_t* spill, int64_t* mean, double* rho, double* alpha, int64_t* bad,
                           uint32_t* status) {
  int64_t nbad = 0;
  memset(n, 0, sizeof(int32_t) * (size_t)R * (size_t)E);
  /* n_re: number of tokens source rank r sends to expert e */
  for (int32_t r = 0; r < R; ++r)
    for (int64_t j = 0; j < N; ++j) {
      int32_t id = ids[(int64_t)r * N + j];
      if (id >= 0 && id < E) n[(int64_t)r * E + id] += 1;
      else nbad += 1;
    }
  /* expert load x_e = sum_r n_re; rank load l_r = sum over its experts */
  for (int32_t e = 0; e < E; ++e) {
    int64_t s = 0;
    for (int32_t r = 0; r < R; ++r) s += n[(int64_t)r * E + e];
    x[e] = s;
  }
  for (int32_t r = 0; r < R; ++r) load[r] = 0;
  for (int32_t e = 0; e < E; ++e) load[home[e]] += x[e];
  int64_t L = 0, lmax = 0;
  for (int32_t r = 0; r < R; ++r) {
    L += load[r];
    if (load[r] > lmax) lmax = load[r];
  }
  int64_t m = L / R;
  for (int32_t r = 0; r < R; ++r) {
    excess[r] = load[r] > m ? load[r] - m : 0;
    spare[r] = m > load[r] ? m - load[r] : 0;
  }
  /* imbalance rho = (max l - mean) / mean with mean = L / R */
  *rho = L > 0 ? (double)((int64_t)R * lmax - L) / (double)L : 0.0;
  /* alpha = mean * R / E = L / E */
  *alpha = (double)L / (double)E;
  *mean = m;
  /* spill: per rank, experts in ascending (load, id) order; sigma_k =
   * max(prefix_k - m, 0); spill of the k-th = sigma_k - sigma_{k-1} */
  int32_t* order = (int32_t*)malloc(sizeof(int32_t) * (size_t)E);
  for (int32_t r = 0; r < R; ++r) {
    int32_t cnt = 0;
    for (int32_t e = 0; e < E; ++e)
      if (home[e] == r) order[cnt++] = e;
    for (int32_t i = 1; i < cnt; ++i) { /* insertion sort by (x asc, e asc) */
      int32_t e = order[i], q = i - 1;
      while (q >= 0 && (x[order[q]] > x[e] || (x[order[q]] == x[e] && order[q] > e))) {
        order[q + 1] = order[q];
        --q;
      }
      order[q + 1] = e;
    }
    int64_t prefix = 0, sigma_prev = 0;
    for (int32_t i = 0; i < cnt; ++i) {
      prefix += x[order[i]];
      int64_t sigma = prefix > m ? prefix - m : 0;
      spill[order[i]] = sigma - sigma_prev;
      sigma_prev = sigma;
    }
  }
  free(order);
  *bad = nbad;
  *status = nbad ? ORACLE_ST_BAD_ID : 0u;
}

int oracle_plan_loads(const int32_t* ids, int32_t B, int32_t R, int64_t N, int32_t E,
                      const int32_t* home, int32_t* n, int64_t* x, int64_t* load, int64_t* excess,
                      int64_t* spare, int64_t* spill, int64_t* mean, double* rho, double* alpha,
                      int64_t* bad, uint32_t* status) {
  if (!ids || !home || !n || !x || !load || !excess || !spare || !spill || !mean || !rho ||
      !alpha || !bad || !status || B < 0 || R <= 0 || N < 0 || E <= 0)
    return -1;
  for (int32_t e = 0; e < E; ++e)
    if (home[e] < 0 || home[e] >= R) return -1;
#pragma omp parallel for schedule(dynamic)
  for (int32_t b = 0; b < B; ++b)
    plan_loads_one(ids + (int64_t)b * R * N, R, N, E, home, n + (int64_t)b * R * E,
                   x + (int64_t)b * E, load + (int64_t)b * R, excess + (int64_t)b * R,
                   spare + (int64_t)b * R, spill + (int64_t)b * E, mean + b, rho + b, alpha + b,
                   bad + b, status + b);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Phase 1 (Sec. A.2): balanced entropic OT by Sinkhorn-Knopp. */

/* log(sum_k exp(t_k)) over the finite terms, with an exact max shift;
 * -inf when no term is finite. */
static double lse(const double* t, int32_t cnt) {
  double mx = -INFINITY;
  for (int32_t k = 0; k < cnt; ++k)
    if (t[k] > mx) mx = t[k];
  if (mx == -INFINITY) return -INFINITY;
  double s = 0.0;
  for (int32_t k = 0; k < cnt; ++k)
    if (t[k] != -INFINITY) s += exp(t[k] - mx);
  return mx + log(s);
}

static double row_residual(const double* s, int32_t R, const double* C, double eps,
                           const double* f, const double* g) {
  double res = 0.0;
  for (int32_t i = 0; i < R; ++i) {
    double rs = 0.0;
    if (f[i] != -INFINITY)
      for (int32_t j = 0; j < R; ++j)
        if (g[j] != -INFINITY) rs += exp((f[i] + g[j] - C[(int64_t)i * R + j]) / eps);
    res += fabs(rs - s[i]);
  }
  return res;
}

/* Column cap (Sec. A.2): scale every column whose mass exceeds its demand
 * back to the demand; columns at or below it are left alone. */
static void column_cap_one(double* T, const double* b, int32_t R) {
  for (int32_t j = 0; j < R; ++j) {
    double c = 0.0;
    for (int32_t i = 0; i < R; ++i) c += T[(int64_t)i * R + j];
    double fac = b[j] / (c + ORACLE_EPS0);
    if (fac > 1.0) fac = 1.0;
    for (int32_t i = 0; i < R; ++i) T[(int64_t)i * R + j] *= fac;
  }
}

static void sinkhorn_one(const double* a, const double* b, int32_t R, const double* C, double eps,
                         int32_t iters, int32_t domain, double tol, int32_t colcap, double* T,
                         double* f, double* g, int32_t* used, uint32_t* status) {
  const int64_t RR = (int64_t)R * R;
  *status = 0;
  *used = 0;
  for (int64_t q = 0; q < RR; ++q) T[q] = 0.0;
  for (int32_t i = 0; i < R; ++i) f[i] = g[i] = -INFINITY;
  int ok = 1;
  for (int32_t i = 0; i < R; ++i) ok &= isfinite(a[i]) && a[i] >= 0.0 && isfinite(b[i]) && b[i] >= 0.0;
  for (int64_t q = 0; q < RR; ++q) ok &= isfinite(C[q]);
  if (!ok) {
    *status = ORACLE_ST_BAD_INPUT;
    return;
  }
  /* supply s = a, demand d = b; equal mass up to the safeguard
   * s~ = gamma * s, gamma = min(1, sum d / max(sum s, eps0)) */
  double S = 0.0, D = 0.0;
  for (int32_t i = 0; i < R; ++i) {
    S += a[i];
    D += b[i];
  }
  if (S <= 0.0 || D <= 0.0) {
    *status = ORACLE_ST_ZERO_MASS;
    return;
  }
  double gamma = D / (S > ORACLE_EPS0 ? S : ORACLE_EPS0);
  if (gamma > 1.0) gamma = 1.0;
  double* s = (double*)malloc(sizeof(double) * (size_t)R);
  double* t = (double*)malloc(sizeof(double) * (size_t)R);
  double mass = 0.0;
  for (int32_t i = 0; i < R; ++i) {
    s[i] = gamma * a[i];
    mass += s[i];
  }

  if (domain == 0) {
    /* log domain: f = eps*log u, g = eps*log v, M = exp(-C/eps):
     *   f_i = eps * (log s_i - LSE_j((g_j - C_ij)/eps))
     *   g_j = eps * (log d_j - LSE_i((f_i - C_ij)/eps))
     * starting from g = 0 (v = 1) on every column. */
    for (int32_t j = 0; j < R; ++j) g[j] = 0.0;
    for (int32_t it = 1; it <= iters; ++it) {
      for (int32_t i = 0; i < R; ++i) {
        if (s[i] > 0.0) {
          for (int32_t j = 0; j < R; ++j)
            t[j] = g[j] == -INFINITY ? -INFINITY : (g[j] - C[(int64_t)i * R + j]) / eps;
          f[i] = eps * (log(s[i]) - lse(t, R));
        } else {
          f[i] = -INFINITY;
        }
      }
      for (int32_t j = 0; j < R; ++j) {
        if (b[j] > 0.0) {
          for (int32_t i = 0; i < R; ++i)
            t[i] = f[i] == -INFINITY ? -INFINITY : (f[i] - C[(int64_t)i * R + j]) / eps;
          g[j] = eps * (log(b[j]) - lse(t, R));
        } else {
          g[j] = -INFINITY;
        }
      }
      *used = it;
      if (tol > 0.0 && row_residual(s, R, C, eps, f, g) <= tol * mass) break;
    }
    /* T = diag(u) M diag(v) = exp((f_i + g_j - C_ij)/eps) */
    for (int32_t i = 0; i < R; ++i)
      for (int32_t j = 0; j < R; ++j)
        if (f[i] != -INFINITY && g[j] != -INFINITY)
          T[(int64_t)i * R + j] = exp((f[i] + g[j] - C[(int64_t)i * R + j]) / eps);
  } else {
    /* linear domain, the GEMV form: u = s / (M v), v = d / (M^T u) */
    double* u = f; /* reuse the output buffers for u and v */
    double* v = g;
    for (int32_t j = 0; j < R; ++j) v[j] = 1.0;
    for (int32_t it = 1; it <= iters; ++it) {
      for (int32_t i = 0; i < R; ++i) {
        double mv = 0.0;
        for (int32_t j = 0; j < R; ++j) mv += exp(-C[(int64_t)i * R + j] / eps) * v[j];
        u[i] = s[i] > 0.0 ? s[i] / mv : 0.0;
      }
      for (int32_t j = 0; j < R; ++j) {
        double mu = 0.0;
        for (int32_t i = 0; i < R; ++i) mu += exp(-C[(int64_t)i * R + j] / eps) * u[i];
        v[j] = b[j] > 0.0 ? b[j] / mu : 0.0;
      }
      *used = it;
      if (tol > 0.0) {
        double res = 0.0;
        for (int32_t i = 0; i < R; ++i) {
          double rs = 0.0;
          for (int32_t j = 0; j < R; ++j) rs += u[i] * exp(-C[(int64_t)i * R + j] / eps) * v[j];
          res += fabs(rs - s[i]);
        }
        if (res <= tol * mass) break;
      }
    }
    for (int32_t i = 0; i < R; ++i)
      for (int32_t j = 0; j < R; ++j)
        T[(int64_t)i * R + j] = u[i] * exp(-C[(int64_t)i * R + j] / eps) * v[j];
    for (int32_t i = 0; i < R; ++i) {
      f[i] = u[i] > 0.0 ? eps * log(u[i]) : -INFINITY;
      g[i] = v[i] > 0.0 ? eps * log(v[i]) : -INFINITY;
    }
  }

  /* column cap, once, on the final plan */
  if (colcap) column_cap_one(T, b, R);
  free(s);
  free(t);
}

int oracle_sinkhorn(const double* a, const double* b, int32_t B, int32_t R, const double* C,
                    int64_t C_stride, double eps, int32_t iters, int32_t domain, double tol,
                    int32_t colcap, double* T, double* f, double* g, int32_t* used,
                    uint32_t* status) {
  if (!a || !b || !C || !T || !f || !g || !used || !status || B < 0 || R <= 0 ||
      !(eps > 0.0) || !isfinite(eps) || iters < 1 || (domain != 0 && domain != 1) ||
      (C_stride != 0 && C_stride != (int64_t)R * R))
    return -1;
#pragma omp parallel for schedule(dynamic)
  for (int32_t p = 0; p < B; ++p)
    sinkhorn_one(a + (int64_t)p * R, b + (int64_t)p * R, R, C + (int64_t)p * C_stride, eps, iters,
                 domain, tol, colcap, T + (int64_t)p * R * R, f + (int64_t)p * R,
                 g + (int64_t)p * R, used + p, status + p);
  return 0;
}

int oracle_column_cap(double* T, const double* b, int32_t B, int32_t R) {
  if (!T || !b || B < 0 || R <= 0) return -1;
  for (int32_t p = 0; p < B; ++p) column_cap_one(T + (int64_t)p * R * R, b + (int64_t)p * R, R);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Topology preference (Sec. A.3 B_er; Sec. A.4 topology bonus). */

int oracle_topology_pref(const float* C, int32_t R, double* Bpref, double* Bauct) {
  if (!C || !Bpref || !Bauct || R <= 0) return -1;
  double cmin = INFINITY;
  for (int32_t i = 0; i < R; ++i)
    for (int32_t j = 0; j < R; ++j) {
      double c = (double)C[(int64_t)i * R + j];
      if (i != j) {
        if (!isfinite(c) || !(c > 0.0)) return -1;
        if (c < cmin) cmin = c;
      }
    }
  if (R == 1) cmin = 1.0;
  for (int32_t i = 0; i < R; ++i)
    for (int32_t j = 0; j < R; ++j) {
      int64_t q = (int64_t)i * R + j;
      if (i == j) {
        Bpref[q] = 0.0;
        Bauct[q] = 1.0;
      } else {
        Bpref[q] = cmin / (double)C[q];
        Bauct[q] = Bpref[q];
      }
    }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Phase 2 (Alg. 2): column-priority iterative matching. */

static void phase2_one(const int64_t* spill, const int64_t* spare, const int64_t* excess,
                       double alpha, const int32_t* home, const float* T, const double* Bpref,
                       int32_t R, int32_t E, int32_t K, uint32_t flags, int32_t* slot_expert,
                       int64_t* slot_amount, int32_t* inner_used) {
  int64_t* spill_p = (int64_t*)malloc(sizeof(int64_t) * (size_t)E);
  int64_t* spare_p = (int64_t*)malloc(sizeof(int64_t) * (size_t)R);
  unsigned char* U = (unsigned char*)calloc((size_t)E * (size_t)R, 1);
  unsigned char* matched = (unsigned char*)malloc((size_t)R);
  int32_t* best_e = (int32_t*)malloc(sizeof(int32_t) * (size_t)R);
  double* best_s = (double*)malloc(sizeof(double) * (size_t)R);
  int32_t* win_r = (int32_t*)malloc(sizeof(int32_t) * (size_t)E);
  double* win_s = (double*)malloc(sizeof(double) * (size_t)E);
  memcpy(spill_p, spill, sizeof(int64_t) * (size_t)E);
  memcpy(spare_p, spare, sizeof(int64_t) * (size_t)R);
  for (int32_t s = 0; s < R * K; ++s) {
    slot_expert[s] = -1;
    slot_amount[s] = 0;
  }
  int32_t nC = 0;
  for (int32_t r = 0; r < R; ++r) nC += spare[r] > 0;
  const double a2 = 0.1 * alpha; /* weight of the OT hint, 0.1 * alpha */
  int32_t used = 0;
  for (int32_t k = 0; k < K; ++k) {
    memset(matched, 0, (size_t)R);
    for (int32_t inner = 0; inner < nC; ++inner) {
      /* Step 1: masked three-level scores; each cold rank picks its best expert */
      int any = 0;
      for (int32_t r = 0; r < R; ++r) {
        best_e[r] = -1;
        best_s[r] = -INFINITY;
        if (matched[r] || spare_p[r] <= 0) continue;
        for (int32_t e = 0; e < E; ++e) {
          int32_t h = home[e];
          if (h == r || U[(int64_t)e * R + r] || spill_p[e] <= 0) continue;
          double q = (double)(spill_p[e] < spare_p[r] ? spill_p[e] : spare_p[r]);
          /* an ablated term (flags) is the literal 0 in the same sum */
          double t1 = (flags & ORACLE_SCH_NO_TOPO) ? 0.0 : alpha * Bpref[(int64_t)h * R + r];
          double ex = (double)excess[h];
          double tn = (double)T[(int64_t)h * R + r] / (ex > ORACLE_EPS0 ? ex : ORACLE_EPS0);
          double t2 = (flags & ORACLE_SCH_NO_FLOW) ? 0.0 : a2 * tn;
          double score = (q + t1) + t2;
          if (score > best_s[r]) { /* strict: lowest e wins ties */
            best_s[r] = score;
            best_e[r] = e;
          }
        }
        any |= best_e[r] >= 0;
      }
      if (!any) break; /* no proposer: the state can no longer change */
      /* Steps 2-3: each proposed expert keeps its best proposer (lowest r on ties) */
      for (int32_t e = 0; e < E; ++e) {
        win_r[e] = -1;
        win_s[e] = -INFINITY;
      }
      for (int32_t r = 0; r < R; ++r) {
        int32_t e = best_e[r];
        if (e >= 0 && best_s[r] > win_s[e]) {
          win_s[e] = best_s[r];
          win_r[e] = r;
        }
      }
      /* Step 4: winners take g = min(spill, spare) into slot k */
      for (int32_t e = 0; e < E; ++e) {
        int32_t r = win_r[e];
        if (r < 0) continue;
        int64_t gq = spill_p[e] < spare_p[r] ? spill_p[e] : spare_p[r];
        spill_p[e] -= gq;
        spare_p[r] -= gq;
        U[(int64_t)e * R + r] = 1;
        matched[r] = 1;
        slot_expert[r * K + k] = e;
        slot_amount[r * K + k] += gq;
      }
      ++used;
    }
  }
  *inner_used = used;
  free(spill_p);
  free(spare_p);
  free(U);
  free(matched);
  free(best_e);
  free(best_s);
  free(win_r);
  free(win_s);
}

/* Row priority (the experts-outer reading of the greedy that Sec. A.3 sets
 * Alg. 2 against): in each slot round k, the experts with spill left are
 * taken in order of their spill at the round's start (largest first, lower
 * id on ties); each in turn takes ranks one at a time, the best-scoring rank
 * with spare left, slot k free and not already holding the expert (same
 * score as Alg. 2, lowest rank on ties), moving min(spill, spare), until its
 * spill is gone or no rank qualifies. */
static const int64_t* g_order_spill; /* sort key of order_cmp */
static int order_cmp(const void* a, const void* b) {
  const int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
  if (g_order_spill[x] != g_order_spill[y]) return g_order_spill[x] > g_order_spill[y] ? -1 : 1;
  return x < y ? -1 : (x > y);
}
static void phase2_row_one(const int64_t* spill, const int64_t* spare, const int64_t* excess,
                           double alpha, const int32_t* home, const float* T, const double* Bpref,
                           int32_t R, int32_t E, int32_t K, uint32_t flags, int32_t* slot_expert,
                           int64_t* slot_amount, int32_t* used_out) {
  int64_t* spill_p = (int64_t*)malloc(sizeof(int64_t) * (size_t)E);
  int64_t* spare_p = (int64_t*)malloc(sizeof(int64_t) * (size_t)R);
  int64_t* key = (int64_t*)malloc(sizeof(int64_t) * (size_t)E);
  int32_t* order = (int32_t*)malloc(sizeof(int32_t) * (size_t)E);
  unsigned char* U = (unsigned char*)calloc((size_t)E * (size_t)R, 1);
  memcpy(spill_p, spill, sizeof(int64_t) * (size_t)E);
  memcpy(spare_p, spare, sizeof(int64_t) * (size_t)R);
  for (int32_t s = 0; s < R * K; ++s) {
    slot_expert[s] = -1;
    slot_amount[s] = 0;
  }
  const double a2 = 0.1 * alpha;
  int32_t used = 0;
  for (int32_t k = 0; k < K; ++k) {
    int32_t n = 0;
    for (int32_t e = 0; e < E; ++e) {
      key[e] = spill_p[e];
      if (spill_p[e] > 0) order[n++] = e;
    }
    g_order_spill = key;
    qsort(order, (size_t)n, sizeof(int32_t), order_cmp);
    for (int32_t i = 0; i < n; ++i) {
      const int32_t e = order[i], h = home[e];
      while (spill_p[e] > 0) {
        int32_t best = -1;
        double bs = -INFINITY;
        for (int32_t r = 0; r < R; ++r) {
          if (spare_p[r] <= 0 || slot_expert[r * K + k] >= 0 || h == r || U[(int64_t)e * R + r]) continue;
          double q = (double)(spill_p[e] < spare_p[r] ? spill_p[e] : spare_p[r]);
          double t1 = (flags & ORACLE_SCH_NO_TOPO) ? 0.0 : alpha * Bpref[(int64_t)h * R + r];
          double ex = (double)excess[h];
          double tn = (double)T[(int64_t)h * R + r] / (ex > ORACLE_EPS0 ? ex : ORACLE_EPS0);
          double t2 = (flags & ORACLE_SCH_NO_FLOW) ? 0.0 : a2 * tn;
          double score = (q + t1) + t2;
          if (score > bs) { /* strict: lowest r wins ties */
            bs = score;
            best = r;
          }
        }
        if (best < 0) break;
        int64_t g = spill_p[e] < spare_p[best] ? spill_p[e] : spare_p[best];
        spill_p[e] -= g;
        spare_p[best] -= g;
        U[(int64_t)e * R + best] = 1;
        slot_expert[best * K + k] = e;
        slot_amount[best * K + k] += g;
        ++used;
      }
    }
  }
  *used_out = used;
  free(spill_p);
  free(spare_p);
  free(key);
  free(order);
  free(U);
}

int oracle_phase2(const int64_t* spill, const int64_t* spare, const int64_t* excess,
                  const double* alpha, const int32_t* home, const float* T, const double* Bpref,
                  int32_t B, int32_t R, int32_t E, int32_t K, uint32_t flags, int32_t* slot_expert,
                  int64_t* slot_amount, int32_t* inner_used) {
  if (!spill || !spare || !excess || !alpha || !home || !T || !Bpref || !slot_expert ||
      !slot_amount || !inner_used || B < 0 || R <= 0 || E <= 0 || K < 0 ||
      (flags & ~(uint32_t)(ORACLE_SCH_NO_TOPO | ORACLE_SCH_NO_FLOW | ORACLE_SCH_ROW_PRIORITY)))
    return -1;
  for (int32_t e = 0; e < E; ++e)
    if (home[e] < 0 || home[e] >= R) return -1;
  if (flags & ORACLE_SCH_ROW_PRIORITY) {
    /* serial over problems: the qsort key is a file-scope pointer */
    for (int32_t b = 0; b < B; ++b)
      phase2_row_one(spill + (int64_t)b * E, spare + (int64_t)b * R, excess + (int64_t)b * R, alpha[b],
                     home, T + (int64_t)b * R * R, Bpref, R, E, K, flags, slot_expert + (int64_t)b * R * K,
                     slot_amount + (int64_t)b * R * K, inner_used + b);
    return 0;
  }
#pragma omp parallel for schedule(dynamic)
  for (int32_t b = 0; b < B; ++b)
    phase2_one(spill + (int64_t)b * E, spare + (int64_t)b * R, excess + (int64_t)b * R, alpha[b],
               home, T + (int64_t)b * R * R, Bpref, R, E, K, flags, slot_expert + (int64_t)b * R * K,
               slot_amount + (int64_t)b * R * K, inner_used + b);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Phase 3 (Alg. 3): Lagrangian auction token assignment. */

static void phase3_one(const int32_t* n, const int32_t* slot_expert, const int64_t* slot_amount,
                       const double* Bauct, int32_t R, int32_t E, int32_t K, double eta,
                       int64_t t_max, int32_t* X, int64_t* unfilled, int64_t* rounds,
                       uint32_t* status) {
  const int32_t S = R * K;
  int64_t* np = (int64_t*)malloc(sizeof(int64_t) * (size_t)R * (size_t)E);
  int64_t* Ap = (int64_t*)malloc(sizeof(int64_t) * (size_t)(S > 0 ? S : 1));
  double* p = (double*)calloc((size_t)R, sizeof(double));
  int32_t* bid = (int32_t*)malloc(sizeof(int32_t) * (size_t)(S > 0 ? S : 1));
  double* bid_s = (double*)malloc(sizeof(double) * (size_t)(S > 0 ? S : 1));
  int32_t* serve = (int32_t*)malloc(sizeof(int32_t) * (size_t)R);
  double* serve_s = (double*)malloc(sizeof(double) * (size_t)R);
  for (int64_t q = 0; q < (int64_t)R * E; ++q) np[q] = n[q];
  for (int32_t s = 0; s < S; ++s) Ap[s] = slot_amount[s];
  for (int64_t q = 0; q < (int64_t)R * S; ++q) X[q] = 0;
  const int64_t tmax = t_max > 0 ? t_max : (int64_t)S * (R + 1);
  int64_t used = 0;
  for (int64_t t = 1; t <= tmax; ++t) {
    /* Step 1: every open slot bids for the source rank maximising B - p */
    int any = 0;
    for (int32_t s = 0; s < S; ++s) {
      bid[s] = -1;
      bid_s[s] = -INFINITY;
      int32_t e = slot_expert[s];
      if (e < 0 || Ap[s] <= 0) continue;
      int32_t host = s / K;
      for (int32_t r = 0; r < R; ++r) {
        if (np[(int64_t)r * E + e] <= 0) continue;
        double sc = Bauct[(int64_t)r * R + host] - p[r];
        if (sc > bid_s[s]) {
          bid_s[s] = sc;
          bid[s] = r;
        }
      }
      any |= bid[s] >= 0;
    }
    if (!any) break;
    /* Step 2: every rank serves its highest-profit bidder (lowest s on ties) */
    for (int32_t r = 0; r < R; ++r) {
      serve[r] = -1;
      serve_s[r] = -INFINITY;
    }
    for (int32_t s = 0; s < S; ++s) {
      int32_t r = bid[s];
      if (r >= 0 && bid_s[s] > serve_s[r]) {
        serve_s[r] = bid_s[s];
        serve[r] = s;
      }
    }
    /* Steps 3-4: transfer x = min(n, A); raise the price of a rank that served */
    for (int32_t r = 0; r < R; ++r) {
      int32_t s = serve[r];
      if (s < 0) continue;
      int32_t e = slot_expert[s];
      int64_t have = np[(int64_t)r * E + e];
      int64_t xq = have < Ap[s] ? have : Ap[s];
      X[(int64_t)r * S + s] += (int32_t)xq;
      np[(int64_t)r * E + e] -= xq;
      Ap[s] -= xq;
      if (xq > 0) p[r] = p[r] + eta;
    }
    used = t;
  }
  int64_t left = 0;
  for (int32_t s = 0; s < S; ++s) left += Ap[s];
  *unfilled = left;
  *rounds = used;
  *status = left > 0 ? ORACLE_ST_UNFILLED : 0u;
  free(np);
  free(Ap);
  free(p);
  free(bid);
  free(bid_s);
  free(serve);
  free(serve_s);
}

int oracle_phase3(const int32_t* n, const int32_t* slot_expert, const int64_t* slot_amount,
                  const double* Bauct, int32_t B, int32_t R, int32_t E, int32_t K, double eta,
                  int64_t t_max, int32_t* X, int64_t* unfilled, int64_t* rounds,
                  uint32_t* status) {
  if (!n || !slot_expert || !slot_amount || !Bauct || !X || !unfilled || !rounds || !status ||
      B < 0 || R <= 0 || E <= 0 || K < 0 || !isfinite(eta))
    return -1;
  for (int64_t q = 0; q < (int64_t)B * R * K; ++q)
    if (slot_expert[q] < -1 || slot_expert[q] >= E || slot_amount[q] < 0) return -1;
#pragma omp parallel for schedule(dynamic)
  for (int32_t b = 0; b < B; ++b)
    phase3_one(n + (int64_t)b * R * E, slot_expert + (int64_t)b * R * K,
               slot_amount + (int64_t)b * R * K, Bauct, R, E, K, eta, t_max,
               X + (int64_t)b * R * R * K, unfilled + b, rounds + b, status + b);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Plan-quality metrics (Sec. 4.1: final imbalance, intra/inter transfers,
 * weighted cost with a 1 : w_inter ratio). */

int oracle_metrics(const int64_t* load, const int32_t* home, const int32_t* slot_expert,
                   const int32_t* X, int32_t B, int32_t R, int32_t E, int32_t K,
                   int32_t ranks_per_node, double w_inter, int64_t* load_after,
                   double* rho_after, int64_t* intra, int64_t* inter, double* weighted) {
  if (!load || !home || !slot_expert || !X || !load_after || !rho_after || !intra || !inter ||
      !weighted || B < 0 || R <= 0 || E <= 0 || K < 0 || ranks_per_node <= 0)
    return -1;
  const int32_t S = R * K;
  for (int32_t b = 0; b < B; ++b) {
    const int64_t* ld = load + (int64_t)b * R;
    int64_t* la = load_after + (int64_t)b * R;
    const int32_t* se = slot_expert + (int64_t)b * S;
    const int32_t* Xb = X + (int64_t)b * R * S;
    int64_t L = 0, lmax = 0, ni = 0, no = 0;
    for (int32_t r = 0; r < R; ++r) {
      la[r] = ld[r];
      L += ld[r];
    }
    for (int32_t s = 0; s < S; ++s) {
      int32_t e = se[s];
      if (e < 0) continue;
      int32_t host = s / K, h = home[e];
      int64_t moved = 0;
      for (int32_t r = 0; r < R; ++r) moved += Xb[(int64_t)r * S + s];
      la[h] -= moved;
      la[host] += moved;
      if (h / ranks_per_node == host / ranks_per_node) ++ni;
      else ++no;
    }
    for (int32_t r = 0; r < R; ++r)
      if (la[r] > lmax) lmax = la[r];
    rho_after[b] = L > 0 ? (double)((int64_t)R * lmax - L) / (double)L : 0.0;
    intra[b] = ni;
    inter[b] = no;
    weighted[b] = (double)ni + w_inter * (double)no;
  }
  return 0;
}

int oracle_max_threads(void) { return omp_get_max_threads(); }
