// C-ABI entry points of libtaot: argument validation, workspace checks and
// kernel launches.  See include/taot.h for the contract of each call.
#include <math.h>

#include "common.h"

using namespace taot;

namespace {

bool bad_dims(int32_t B, int32_t R) { return B < 0 || R <= 0; }

}  // namespace

extern "C" {

const char* taot_status_string(taot_status s) {
  switch (s) {
    case TAOT_OK: return "ok";
    case TAOT_ERR_INVALID_ARG: return "invalid argument";
    case TAOT_ERR_UNSUPPORTED: return "unsupported shape";
    case TAOT_ERR_WORKSPACE: return "workspace missing or too small";
    case TAOT_ERR_LAUNCH: return "kernel launch failed";
    case TAOT_ERR_SCRATCH: return "needs more than the fixed scratch of the allocation-free entry point";
  }
  return "unknown status";
}

size_t taot_plan_loads_workspace_size(int32_t B, int32_t R, int32_t E) {
  if (bad_dims(B, R) || E <= 0) return 0;
  return plan_loads_ws(B, R, E);
}

taot_status taot_plan_loads(const int32_t* ids, int32_t B, int32_t R, int64_t N, int32_t E,
                            const int32_t* home, int32_t* n, int64_t* load_e, int64_t* load_r,
                            int64_t* excess, int64_t* spare, int64_t* spill, float* supply,
                            float* demand, double* rho, double* alpha, int64_t* bad_ids,
                            int32_t* hot_idx, int32_t* cold_idx, int32_t* hot_cnt, int32_t* cold_cnt,
                            uint32_t* status, void* ws, size_t ws_bytes, void* stream) {
  if (bad_dims(B, R) || E <= 0 || N < 0) return TAOT_ERR_INVALID_ARG;
  if (R > TAOT_MAX_RANKS || E > TAOT_MAX_EXPERTS) return TAOT_ERR_UNSUPPORTED;
  if (B == 0) return TAOT_OK;
  if ((N > 0 && !ids) || !home || !n || !load_e || !load_r || !excess || !spare || !spill || !alpha)
    return TAOT_ERR_INVALID_ARG;
  if ((int64_t)B * R > 0x7fffffffLL || N > 0x7fffffffLL) return TAOT_ERR_UNSUPPORTED;
  if (!ws || ws_bytes < plan_loads_ws(B, R, E)) return TAOT_ERR_WORKSPACE;
  return launch_plan_loads(ids, B, R, N, E, home, n, load_e, load_r, excess, spare, spill, supply,
                           demand, rho, alpha, bad_ids, hot_idx, cold_idx, hot_cnt, cold_cnt, status, ws,
                           static_cast<hipStream_t>(stream));
}

taot_status taot_plan_loads_noalloc(const int32_t* ids, int32_t B, int32_t R, int64_t N, int32_t E,
                                    const int32_t* home, int32_t* n, int64_t* load_e, int64_t* load_r,
                                    int64_t* excess, int64_t* spare, int64_t* spill, float* supply,
                                    float* demand, double* rho, double* alpha, int64_t* bad_ids,
                                    int32_t* hot_idx, int32_t* cold_idx, int32_t* hot_cnt, int32_t* cold_cnt,
                                    uint32_t* status, void* stream) {
  if (bad_dims(B, R) || E <= 0 || N < 0) return TAOT_ERR_INVALID_ARG;
  if (R > TAOT_MAX_RANKS || E > TAOT_MAX_EXPERTS) return TAOT_ERR_UNSUPPORTED;
  if (B == 0) return TAOT_OK;
  if ((N > 0 && !ids) || !home || !n || !load_e || !load_r || !excess || !spare || !spill || !alpha)
    return TAOT_ERR_INVALID_ARG;
  if ((int64_t)B * R > 0x7fffffffLL || N > 0x7fffffffLL) return TAOT_ERR_UNSUPPORTED;
  if (plan_loads_ws(B, R, E) > plan_loads_scratch_limit()) return TAOT_ERR_SCRATCH;
  void* ws = plan_loads_scratch();
  if (!ws) return TAOT_ERR_LAUNCH;
  return launch_plan_loads(ids, B, R, N, E, home, n, load_e, load_r, excess, spare, spill, supply,
                           demand, rho, alpha, bad_ids, hot_idx, cold_idx, hot_cnt, cold_cnt, status, ws,
                           static_cast<hipStream_t>(stream));
}

size_t taot_plan_loads_noalloc_max_problems(int32_t R, int32_t E) {
  if (R <= 0 || E <= 0 || R > TAOT_MAX_RANKS || E > TAOT_MAX_EXPERTS) return 0;
  size_t lo = 0, hi = (size_t)1 << 31;  // largest B whose workspace fits the scratch
  while (lo + 1 < hi) {
    const size_t mid = (lo + hi) / 2;
    if (plan_loads_ws((int32_t)(mid > 0x7fffffff ? 0x7fffffff : mid), R, E) <= plan_loads_scratch_limit()) lo = mid;
    else hi = mid;
  }
  return lo;
}

size_t taot_sinkhorn_workspace_size(int32_t B, int32_t R) {
  if (bad_dims(B, R)) return 0;
  return sinkhorn_ws(B, R);
}

taot_status taot_sinkhorn_batched(const float* a, const float* b, int32_t B, int32_t R,
                                  const float* C, int64_t C_batch_stride, float eps,
                                  int32_t iters, uint32_t flags, float* T, float* f, float* g,
                                  uint32_t* status, void* ws, size_t ws_bytes, void* stream) {
  if (bad_dims(B, R) || !(eps > 0.f) || !isfinite(eps) || iters < 1 ||
      (C_batch_stride != 0 && C_batch_stride != (int64_t)R * R) ||
      (flags & ~(TAOT_SK_NO_COLCAP | TAOT_SK_FORCE_STREAM | TAOT_SK_NO_REGISTER | TAOT_SK_WAVES_1 |
                 TAOT_SK_DENSE | TAOT_SK_LINEAR)))
    return TAOT_ERR_INVALID_ARG;
  if (R > TAOT_MAX_RANKS) return TAOT_ERR_UNSUPPORTED;
  if (B == 0) return TAOT_OK;
  if (!a || !b || !C) return TAOT_ERR_INVALID_ARG;
  if (!ws || ws_bytes < sinkhorn_ws(B, R)) return TAOT_ERR_WORKSPACE;
  return launch_sinkhorn(a, b, B, R, C, C_batch_stride, eps, iters, flags, T, f, g, status, ws,
                         static_cast<hipStream_t>(stream));
}

size_t taot_round_schedule_workspace_size(int32_t B, int32_t R, int32_t E, int32_t K) {
  if (bad_dims(B, R) || E <= 0 || K < 0) return 0;
  return schedule_ws(B, R, E, K);
}

taot_status taot_round_schedule(const int32_t* n, const int64_t* spill, const int64_t* spare,
                                const int64_t* excess, const double* alpha, const int32_t* home,
                                const float* T, const double* Bpref, const double* Bauct,
                                int32_t B, int32_t R, int32_t E, int32_t K, double price_step,
                                int64_t t_max, uint32_t flags, int32_t* slot_expert, int64_t* slot_amount,
                                int32_t* X, int64_t* unfilled, int32_t* rounds_used,
                                uint32_t* status, void* ws, size_t ws_bytes, void* stream) {
  if (bad_dims(B, R) || E <= 0 || K < 0 || !isfinite(price_step)) return TAOT_ERR_INVALID_ARG;
  if (flags & ~(TAOT_SCH_NO_TOPO | TAOT_SCH_NO_FLOW | TAOT_SCH_ROW_PRIORITY)) return TAOT_ERR_INVALID_ARG;
  if (R > TAOT_MAX_RANKS || E > TAOT_MAX_EXPERTS || K > TAOT_MAX_SLOTS_PER_RANK)
    return TAOT_ERR_UNSUPPORTED;
  if (B == 0) return TAOT_OK;
  if (!n || !spill || !spare || !excess || !alpha || !home || !T || !Bpref || !Bauct ||
      (K > 0 && (!slot_expert || !slot_amount || !X)) || !unfilled)
    return TAOT_ERR_INVALID_ARG;
  if ((int64_t)R * K * R > 0x7fffffffLL * 8) return TAOT_ERR_UNSUPPORTED;
  if (!ws || ws_bytes < schedule_ws(B, R, E, K)) return TAOT_ERR_WORKSPACE;
  return launch_schedule(n, spill, spare, excess, alpha, home, T, Bpref, Bauct, B, R, E, K,
                         price_step, t_max, flags, slot_expert, slot_amount, X, unfilled, rounds_used,
                         status, ws, static_cast<hipStream_t>(stream));
}

taot_status taot_topology_pref(const float* C_host, int32_t R, double* Bpref_host,
                               double* Bauct_host) {
  if (!C_host || !Bpref_host || !Bauct_host || R <= 0) return TAOT_ERR_INVALID_ARG;
  double cmin = INFINITY;
  for (int64_t i = 0; i < R; ++i)
    for (int64_t j = 0; j < R; ++j) {
      if (i == j) continue;
      const double c = (double)C_host[i * R + j];
      if (!isfinite(c) || !(c > 0.0)) return TAOT_ERR_INVALID_ARG;
      cmin = c < cmin ? c : cmin;
    }
  if (R == 1) cmin = 1.0;
  for (int64_t i = 0; i < R; ++i)
    for (int64_t j = 0; j < R; ++j) {
      const int64_t q = i * R + j;
      if (i == j) {
        Bpref_host[q] = 0.0;
        Bauct_host[q] = 1.0;
      } else {
        Bpref_host[q] = cmin / (double)C_host[q];
        Bauct_host[q] = Bpref_host[q];
      }
    }
  return TAOT_OK;
}

}  // extern "C"
