/* libtaot: MI355X (gfx950) implementation of the TAOT per-step replica planner.
 *
 * Reference: "TAOT: Topology-Aware Optimal Transport for Dynamic Expert Replica
 * Placement in MoE Training" (arXiv 2608.03676), Sec. 3 and Appendix A.
 *
 * Conventions for every entry point
 *   - Arrays are contiguous, row-major DEVICE pointers unless marked "host".
 *   - The caller owns every input, output and workspace buffer.  The library
 *     never allocates, frees or keeps pointers and has no mutable global state
 *     (one exception: the fixed device scratch of taot_plan_loads_noalloc);
 *     calls on different streams may run concurrently.
 *   - Each call only enqueues work on `stream` (a hipStream_t; 0 = the null
 *     stream) and returns without synchronising.  Every output is fully
 *     overwritten by the enqueued work.
 *   - Errors the host can detect (null pointers, bad sizes, undersized
 *     workspace, unsupported shapes) return a non-zero taot_status and enqueue
 *     nothing.  Conditions found in the data set bits of the per-problem
 *     `status` array (TAOT_ST_*), which the caller reads after synchronising;
 *     device code never aborts.
 *   - Workspace: pass at least taot_*_workspace_size(...) bytes, 256-byte
 *     aligned (hipMalloc and torch allocations are).
 */
#ifndef TAOT_H
#define TAOT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TAOT_OK = 0,
  TAOT_ERR_INVALID_ARG = 1, /* null pointer, negative size, eps <= 0, ...      */
  TAOT_ERR_UNSUPPORTED = 2, /* shape beyond the limits below                    */
  TAOT_ERR_WORKSPACE = 3,   /* ws == NULL or ws_bytes < the required size      */
  TAOT_ERR_LAUNCH = 4,      /* the HIP runtime rejected a kernel launch        */
  TAOT_ERR_SCRATCH = 5,     /* taot_plan_loads_noalloc: the shape needs more than
                               its fixed scratch (see there)                   */
} taot_status;

/* Per-problem status bits (uint32_t status[B]). */
#define TAOT_ST_BAD_ID 0x1u    /* plan_loads: routing ids outside [0, E) were skipped   */
#define TAOT_ST_BAD_INPUT 0x2u /* plan_loads: a home rank outside [0, R); sinkhorn: an
                                  entry of a or b negative or non-finite, or any of
                                  the R*R entries of the problem's C non-finite; the
                                  problem's outputs are zero (f, g = -inf)          */
#define TAOT_ST_ZERO_MASS 0x4u /* sinkhorn: total supply or demand is zero; T = 0      */
#define TAOT_ST_UNFILLED 0x8u  /* round_schedule: the auction stopped at t_max with
                                  planned tokens left unassigned (`unfilled` > 0)   */
#define TAOT_ST_STREAMED 0x10u /* sinkhorn (informational): the plan block did not fit
                                  on chip and was streamed through device memory    */

/* Shape limits (TAOT_ERR_UNSUPPORTED beyond them). */
#define TAOT_MAX_RANKS 2048
#define TAOT_MAX_EXPERTS 32768
#define TAOT_MAX_SLOTS_PER_RANK 64

/* Sinkhorn flags. */
#define TAOT_SK_NO_COLCAP 0x1u    /* skip the column-cap safeguard                      */
#define TAOT_SK_FORCE_STREAM 0x2u /* keep the plan block in device memory even when it
                                     would fit on chip (exercises the large-R path)  */
#define TAOT_SK_NO_REGISTER 0x4u  /* do not use the register-resident path
                                     (exercises the LDS-resident path)               */
#define TAOT_SK_WAVES_1 0x8u      /* run each register-resident problem on one wave
                                     where its rows fit one wave's registers (by
                                     default small batches spread a problem over
                                     up to four waves)                              */
#define TAOT_SK_DENSE 0x10u       /* dense streamed iterate (Sec. A.2, GEMV form): the
                                     stabilised updates over all R x R entries of
                                     every problem, with no support compaction; each
                                     iteration streams the stored kernel matrix
                                     (built from C in the first) from device memory
                                     through every compute unit.  Same outputs as
                                     the default paths (to rounding); status
                                     TAOT_ST_STREAMED.  The other TAOT_SK_* flags
                                     except NO_COLCAP and LINEAR are ignored      */
#define TAOT_SK_LINEAR 0x20u      /* the linear-domain GEMV form itself (Sec. A.2):
                                     u = s~ / (M v), v = d / (M^T u) with
                                     M = exp(-C / eps) formed once in fp32 and no
                                     stabilisation, on the dense streamed kernels
                                     (implies TAOT_SK_DENSE).  Valid only while M's
                                     entries and the scalings stay in fp32's normal
                                     range (costs up to about 80 eps); beyond it the
                                     plan may hold zeros, inf or NaN, as the plain
                                     form does                                     */

/* round_schedule flags: ablations of the Phase-2 score (Sec. A.3 discusses
 * the contribution of each term).  Phase 3 is unaffected. */
#define TAOT_SCH_NO_TOPO 0x1u  /* drop the topology term alpha * Bpref (score q + 0.1 alpha Tn) */
#define TAOT_SCH_NO_FLOW 0x2u  /* drop the flow-hint term 0.1 * alpha * Tn (score q + alpha Bpref) */
#define TAOT_SCH_ROW_PRIORITY 0x4u /* Phase 2 from the experts' side (the greedy Sec. A.3 sets
                                      Alg. 2 against): each slot round takes the experts with
                                      spill left by spill at the round's start (largest first,
                                      lower id on ties), and each takes its best-scoring ranks
                                      with spare left and the slot free, one at a time (lowest
                                      rank on ties), until its spill is gone; rounds_used[b][0]
                                      then counts placements */

/* Returns a static description of a status code (host, never NULL). */
const char* taot_status_string(taot_status s);

/* ------------------------------------------------------------------------ */
/* Steps 1-2: expert-load histogram, rank loads, overload/spare marginals and
 * spill (Sec. 3.1 "Problem Formulation"; Sec. A.1 load, excess/spare, rho and
 * hot/cold definitions; Sec. A.3 spill by cumulative-excess differencing).
 *
 *   ids     [B][R][N] int32   expert chosen by each routed token, grouped by the
 *                             source rank r that sends it (N = tokens * top-k);
 *                             ids outside [0, E) are skipped and counted.
 *   home    [E]       int32   home rank of each expert (any map into [0, R)).
 * Outputs:
 *   n       [B][R][E] int32   n_re, tokens rank r sends to expert e.  The call
 *                             also stages the counts here (16-bit pairs for
 *                             rows of fewer than 2 * 65535 ids), so n holds
 *                             n_re only once the call's work on `stream` has
 *                             finished, and not after TAOT_ERR_LAUNCH.
 *   load_e  [B][E]    int64   expert load x_e = sum_r n_re.
 *   load_r  [B][R]    int64   rank load l_r = sum of x_e over its experts.
 *   excess  [B][R]    int64   max(l_r - m, 0) with the integer mean m = floor(L/R),
 *   spare   [B][R]    int64   max(m - l_r, 0);  L = sum_r l_r.
 *   spill   [B][E]    int64   per rank, experts in ascending (x_e, e) order, spill =
 *                             sigma_k - sigma_{k-1}, sigma_k = max(prefix_k - m, 0).
 *   supply  [B][R]    float   excess as fp32 (Sinkhorn supply s), nullable.
 *   demand  [B][R]    float   spare as fp32 (Sinkhorn demand d), nullable.
 *   rho     [B]       double  imbalance (max_r l_r - L/R) / (L/R) (0 if L = 0), nullable.
 *   alpha   [B]       double  score scale alpha = mean * R / E = L / E.
 *   bad_ids [B]       int64   ids outside [0, E), nullable.
 *   hot_idx [B][R]    int32   the hot set H = {r : l_r > m} in ascending rank
 *                             order, then -1 (nullable);
 *   cold_idx [B][R]   int32   the cold set C = {r : l_r < m} likewise (nullable);
 *   hot_cnt, cold_cnt [B] int32  |H| and |C| (each nullable).  The Sinkhorn
 *                             derives its support from a and b itself, so
 *                             these are outputs for the caller only.
 *   status  [B]       uint32  TAOT_ST_BAD_ID, TAOT_ST_BAD_INPUT (home out of range).
 * Limits: 1 <= R <= TAOT_MAX_RANKS, 1 <= E <= TAOT_MAX_EXPERTS, B >= 0,
 * 0 <= N <= 2^31 - 1 and B * R <= 2^31 - 1 (else TAOT_ERR_UNSUPPORTED).
 */
size_t taot_plan_loads_workspace_size(int32_t B, int32_t R, int32_t E);
taot_status taot_plan_loads(const int32_t* ids, int32_t B, int32_t R, int64_t N, int32_t E,
                            const int32_t* home, int32_t* n, int64_t* load_e, int64_t* load_r,
                            int64_t* excess, int64_t* spare, int64_t* spill, float* supply,
                            float* demand, double* rho, double* alpha, int64_t* bad_ids,
                            int32_t* hot_idx, int32_t* cold_idx, int32_t* hot_cnt, int32_t* cold_cnt,
                            uint32_t* status, void* ws, size_t ws_bytes, void* stream);

/* Allocation-free variant of taot_plan_loads, for callers that cannot
 * allocate device memory or pass a workspace (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation).  Same arguments,
 * outputs and status bits as taot_plan_loads without ws / ws_bytes; the
 * enqueued kernels are the same.  Its workspace is a fixed 1 MiB array in
 * device memory of the library, one per GPU, set up on the first call on
 * each device and kept until the process ends; no call allocates or frees
 * memory.  Every call on one GPU uses the same array (its contents are
 * rebuilt by each call), so calls that overlap on one GPU, on different
 * streams or host threads, race: serialise them.
 * Returns TAOT_ERR_SCRATCH, enqueuing nothing, when the shape's workspace
 * exceeds the array: B above taot_plan_loads_noalloc_max_problems(R, E)
 * (about 1.1e5 problems at R = 2048, E = 32768), TAOT_ERR_LAUNCH if the
 * array's device address cannot be obtained. */
taot_status taot_plan_loads_noalloc(const int32_t* ids, int32_t B, int32_t R, int64_t N, int32_t E,
                                    const int32_t* home, int32_t* n, int64_t* load_e, int64_t* load_r,
                                    int64_t* excess, int64_t* spare, int64_t* spill, float* supply,
                                    float* demand, double* rho, double* alpha, int64_t* bad_ids,
                                    int32_t* hot_idx, int32_t* cold_idx, int32_t* hot_cnt, int32_t* cold_cnt,
                                    uint32_t* status, void* stream);
/* Largest B taot_plan_loads_noalloc accepts for R ranks and E experts (0 for
 * an invalid or unsupported R or E). */
size_t taot_plan_loads_noalloc_max_problems(int32_t R, int32_t E);

/* ------------------------------------------------------------------------ */
/* Step 3: batched Phase-1 Sinkhorn-Knopp flow planning (Sec. 3.2 "Phase 1";
 * Sec. A.2: balanced entropic OT, Gibbs form diag(u) M diag(v) with
 * M = exp(-C/eps), the alternating u/v updates, supply scaling gamma and the
 * column-cap safeguard).
 *
 * For every problem b: s~ = gamma * a_b with gamma = min(1, sum b_b /
 * max(sum a_b, 1e-12)); starting from v = 1 on all R columns, `iters`
 * iterations of u = s~ / (M v) then v = d / (M^T u); T = diag(u) M diag(v);
 * then (unless TAOT_SK_NO_COLCAP) T_ij *= min(1, d_j / (sum_i T_ij + 1e-12)).
 * The iterate is computed in fp32 with log-domain stabilisation, so it matches
 * the double-precision definition to rounding (not bit for bit).
 *
 *   a, b    [B][R] float   supply and demand (non-negative, finite).
 *   C       [R][R] float   cost; C_batch_stride = 0 shares one matrix, R*R gives
 *                          one per problem.  Any real values; every entry is
 *                          checked, and a NaN or infinity anywhere in a
 *                          problem's matrix marks that problem BAD_INPUT.
 *   eps     > 0            absolute entropic regulariser.
 *   iters   >= 1           Sinkhorn iterations (one iteration = u then v update).
 *   flags   TAOT_SK_*.
 * Outputs (each nullable):
 *   T       [B][R][R] float  plan; zero outside supp(a) x supp(b).
 *   f, g    [B][R]    float  potentials eps*log u, eps*log v (-inf off the support).
 *   status  [B]       uint32 TAOT_ST_BAD_INPUT, TAOT_ST_ZERO_MASS, TAOT_ST_STREAMED.
 * Limits: 1 <= R <= TAOT_MAX_RANKS.
 */
size_t taot_sinkhorn_workspace_size(int32_t B, int32_t R);
taot_status taot_sinkhorn_batched(const float* a, const float* b, int32_t B, int32_t R,
                                  const float* C, int64_t C_batch_stride, float eps,
                                  int32_t iters, uint32_t flags, float* T, float* f, float* g,
                                  uint32_t* status, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Steps 4-5: integer replica matching and token split (Sec. 3.2 "Phase 2" and
 * "Phase 3"; Alg. 2 column-priority iterative matching with the three-level
 * score of Sec. A.3; Alg. 3 Lagrangian auction of Sec. A.4).
 *
 * Slots: s = r*K + k (k < K) is guest slot k of rank r (S = R*K).
 * Phase 2 score of expert e on rank r, evaluated in fp64 in this order with
 * every operation rounded (no fused multiply-add):
 *     ((q + alpha * Bpref[home(e)][r]) + (0.1 * alpha) * Tn)
 *     q  = min(spill'_e, spare'_r),  Tn = T[home(e)][r] / max(excess[home(e)], 1e-12)
 * Every argmax is masked to its candidates and breaks ties to the lowest index.
 * Phase 3 runs rounds of: each open slot bids for the source rank with tokens
 * of its expert maximising Bauct[r][host(s)] - p_r; each rank serves its best
 * bidder with min(n'_{r,e}, A'_s) tokens and raises its price by price_step;
 * it stops after the first round without a bid or after t_max rounds.
 *
 *   n       [B][R][E] int32   token counts (from taot_plan_loads).
 *   spill   [B][E], spare [B][R], excess [B][R] int64 and alpha [B] double
 *                             (from taot_plan_loads).
 *   home    [E]       int32   home ranks.
 *   T       [B][R][R] float   Phase-1 plan (from taot_sinkhorn_batched).
 *   Bpref   [R][R]    double  Phase-2 topology preference (0 on the diagonal).
 *   Bauct   [R][R]    double  Phase-3 topology bonus.
 *   K       0..TAOT_MAX_SLOTS_PER_RANK guest slots per rank.
 *   price_step  finite, the auction's price increment.
 *   t_max   maximum auction rounds; <= 0 selects R*K*(R+1).
 *   flags   TAOT_SCH_* (0 for the method as published): a dropped term
 *           enters the score as +0 in the same evaluation order.
 * Outputs:
 *   slot_expert [B][R*K] int32   expert placed in slot s, -1 if empty.
 *   slot_amount [B][R*K] int64   tokens planned for slot s (A).
 *   X           [B][R][R*K] int32  tokens source rank r sends to slot s.
 *   unfilled    [B] int64          planned tokens left unassigned.
 *   rounds_used [B][2] int32       Phase-2 inner iterations, Phase-3 rounds
 *                                  (nullable, diagnostic).
 *   status      [B] uint32         TAOT_ST_UNFILLED, TAOT_ST_BAD_INPUT.
 * Bit-exact with a double-precision reference that follows the same order.
 */
size_t taot_round_schedule_workspace_size(int32_t B, int32_t R, int32_t E, int32_t K);
taot_status taot_round_schedule(const int32_t* n, const int64_t* spill, const int64_t* spare,
                                const int64_t* excess, const double* alpha, const int32_t* home,
                                const float* T, const double* Bpref, const double* Bauct,
                                int32_t B, int32_t R, int32_t E, int32_t K, double price_step,
                                int64_t t_max, uint32_t flags, int32_t* slot_expert, int64_t* slot_amount,
                                int32_t* X, int64_t* unfilled, int32_t* rounds_used,
                                uint32_t* status, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Host helper: topology-preference matrices from a cost matrix (Sec. A.3
 * topology preference B: 1 intra-node, w_inter < 1 inter-node, 0 for the home
 * rank; Sec. A.4 topology bonus).  With cmin the smallest off-diagonal cost:
 *   Bpref[i][j] = cmin / C[i][j] (i != j), 0 (i == j);
 *   Bauct[i][j] = Bpref[i][j]    (i != j), 1 (i == j).
 * All pointers are HOST pointers ([R][R]); off-diagonal costs must be finite
 * and > 0.  Returns TAOT_ERR_INVALID_ARG otherwise. */
taot_status taot_topology_pref(const float* C_host, int32_t R, double* Bpref_host,
                               double* Bauct_host);

#ifdef __cplusplus
}
#endif
#endif /* TAOT_H */
