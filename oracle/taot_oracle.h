/* Reference oracle for the TAOT per-step replica planner.
 *
 * TEST INFRASTRUCTURE ONLY.  Plain, slow, double-precision C that follows the
 * paper's definitions and algorithms step by step.  Only the tests, the
 * package's smoke() entry and the benchmark's CPU-baseline leg may call it;
 * the planner library never does.  It shares no code with the GPU library.
 *
 * All arrays are host arrays, row-major, owned by the caller.  Every entry
 * point loops over problems b in [0, B) (OpenMP) and returns 0, or -1 for
 * invalid arguments (nothing written).
 *
 * Parity status: every function is pinned by the CPU tests (closed forms,
 * invariants, brute force, hand-traced cases) except where the header of the
 * .c file says "parity unpinned".
 */
#ifndef TAOT_ORACLE_H
#define TAOT_ORACLE_H
#include <stdint.h>

#define ORACLE_EPS0 1e-12
/* Phase-2 score ablations: drop alpha * Bpref, or drop 0.1 * alpha * Tn */
#define ORACLE_SCH_NO_TOPO 0x1u
#define ORACLE_SCH_NO_FLOW 0x2u
/* Phase-2 matching from the experts' side (row priority) instead of Alg. 2 */
#define ORACLE_SCH_ROW_PRIORITY 0x4u

#define ORACLE_ST_BAD_ID 1u
#define ORACLE_ST_BAD_INPUT 2u
#define ORACLE_ST_ZERO_MASS 4u
#define ORACLE_ST_UNFILLED 8u

#ifdef __cplusplus
extern "C" {
#endif

/* Threads the OpenMP loops over problems may use (omp_get_max_threads). */
int oracle_max_threads(void);

/* Sec. 3.1 / A.1: expert-load histogram, rank loads, excess/spare, rho,
 * alpha and the spill of Sec. A.3.
 *   ids   [B][R][N] int32 routing ids (expert chosen by a token of source rank r)
 *   home  [E]       home rank of each expert
 * outputs (all [B]-major): n [B][R][E], x [B][E], load [B][R], excess [B][R],
 *   spare [B][R], spill [B][E], mean [B] (floor(L/R)), rho [B], alpha [B],
 *   bad [B] (ids outside [0,E)), status [B]. */
int oracle_plan_loads(const int32_t* ids, int32_t B, int32_t R, int64_t N, int32_t E,
                      const int32_t* home, int32_t* n, int64_t* x, int64_t* load, int64_t* excess,
                      int64_t* spare, int64_t* spill, int64_t* mean, double* rho, double* alpha,
                      int64_t* bad, uint32_t* status);

/* Sec. A.2: entropic OT between supply a and demand b under cost C.
 *   a, b [B][R] (non-negative), C [R][R] with batch stride C_stride (0 or R*R)
 *   eps > 0, iters >= 1.
 *   domain 0: log domain with an exact max-shifted log-sum-exp (reference);
 *   domain 1: the plain linear-domain scaling updates u = s/(Mv), v = d/(M^T u).
 *   tol > 0: run to tolerance instead, i.e. stop after the first iteration whose
 *            row residual sum_i |sum_j T_ij - s~_i| <= tol * mass (iters is the cap).
 *   colcap != 0 applies the column-cap safeguard once after the last iteration.
 * outputs: T [B][R][R], f [B][R], g [B][R] (natural-log potentials eps*log u,
 *   eps*log v; -inf off the support), used [B] iterations run, status [B]. */
int oracle_sinkhorn(const double* a, const double* b, int32_t B, int32_t R, const double* C,
                    int64_t C_stride, double eps, int32_t iters, int32_t domain, double tol,
                    int32_t colcap, double* T, double* f, double* g, int32_t* used,
                    uint32_t* status);

/* Topology-preference matrices derived from C (fp32 input, fp64 output):
 *   Bpref[i][j] = cmin / C[i][j] for i != j (cmin = smallest off-diagonal cost), 0 on i == j;
 *   Bauct[i][j] = Bpref[i][j] for i != j, 1 on i == j. */
/* The column-cap safeguard of Sec. A.2 on its own, in place on B plans
 * T [B][R][R] with demands b [B][R]: c_j = sum_i T_ij, then
 * T_ij <- T_ij * min(1, b_j / (c_j + eps0)).  oracle_sinkhorn applies this
 * same step to its final plan when colcap != 0. */
int oracle_column_cap(double* T, const double* b, int32_t B, int32_t R);

int oracle_topology_pref(const float* C, int32_t R, double* Bpref, double* Bauct);

/* Alg. 2 (Phase 2, column-priority matching) for B problems.
 *   T [B][R][R] is the Phase-1 plan in fp32 (promoted to fp64 inside).
 *   flags: ORACLE_SCH_* ablations of the score (0 for the method as published);
 *   ORACLE_SCH_ROW_PRIORITY replaces Alg. 2 by the experts-outer greedy that
 *   Sec. A.3 contrasts it with (inner_used then counts placements).
 * outputs: slot_expert [B][R*K] (-1 empty), slot_amount [B][R*K],
 *   inner_used [B] (inner iterations executed, summed over rounds). */
int oracle_phase2(const int64_t* spill, const int64_t* spare, const int64_t* excess,
                  const double* alpha, const int32_t* home, const float* T, const double* Bpref,
                  int32_t B, int32_t R, int32_t E, int32_t K, uint32_t flags, int32_t* slot_expert,
                  int64_t* slot_amount, int32_t* inner_used);

/* Alg. 3 (Phase 3, Lagrangian auction) for B problems.
 *   n [B][R][E] token counts, slots from Phase 2, Bauct [R][R], price step eta,
 *   t_max (<= 0: R*K*(R+1)).
 * outputs: X [B][R][R*K], unfilled [B], rounds [B], status [B] (UNFILLED bit). */
int oracle_phase3(const int32_t* n, const int32_t* slot_expert, const int64_t* slot_amount,
                  const double* Bauct, int32_t B, int32_t R, int32_t E, int32_t K, double eta,
                  int64_t t_max, int32_t* X, int64_t* unfilled, int64_t* rounds,
                  uint32_t* status);

/* Plan-quality metrics of Sec. 4.1 for one schedule per problem:
 *   post-plan rank loads load_after [B][R], rho_after [B], intra/inter replica
 *   counts [B] (node = rank / ranks_per_node) and the weighted cost
 *   intra + w_inter * inter [B]. */
int oracle_metrics(const int64_t* load, const int32_t* home, const int32_t* slot_expert,
                   const int32_t* X, int32_t B, int32_t R, int32_t E, int32_t K,
                   int32_t ranks_per_node, double w_inter, int64_t* load_after,
                   double* rho_after, int64_t* intra, int64_t* inter, double* weighted);

#ifdef __cplusplus
}
#endif
#endif
