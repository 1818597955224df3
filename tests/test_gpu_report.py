"""The per-invocation planner report (Appendix B.3: load before routing,
the cloning plan, the projected load, the summary) from a plan made on the
device equals the report made from the oracle's own outputs, line for line.
The device plan's schedule consumes the oracle's plan cast to fp32, as in
every schedule parity test, so both sides hold the same integers."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2608_03676_amd as taot
import workloads as W
from helpers import oracle_inputs

pytestmark = pytest.mark.gpu


def _oracle_plan(w, ids, L, C, K):
    """The oracle's plan in the binding's dataclasses (CPU tensors)."""
    P = O.sinkhorn(L.excess.astype(float), L.spare.astype(float), C.astype(float), w.eps, w.iters)
    Bp, Ba = O.topology_pref(C)
    home = W.home_map(w)
    T32 = P.T.astype(np.float32)
    se, sa, _ = O.phase2(L.spill, L.spare, L.excess, L.alpha, home, T32, Bp, K)
    X, unfilled, _, st = O.phase3(L.n, se, sa, Ba, K, w.price_step)
    t = torch.from_numpy
    B = ids.shape[0]
    loads = taot.Loads(t(L.n), t(L.x), t(L.load), t(L.excess), t(L.spare), t(L.spill),
                       t(L.excess.astype(np.float32)), t(L.spare.astype(np.float32)), t(L.rho), t(L.alpha),
                       t(L.bad), t(L.status.view(np.int32)))
    flow = taot.Flow(t(T32), t(P.f.astype(np.float32)), t(P.g.astype(np.float32)), torch.zeros(B, dtype=torch.int32))
    sched = taot.Schedule(t(se), t(sa), t(X), t(unfilled), torch.zeros((B, 2), dtype=torch.int32),
                          t(st.view(np.int32)))
    return taot.Plan(loads, flow, sched), T32


@pytest.mark.parametrize("cfg,problems,K", [(0, [0], 2), (1, [0, 1, 2], 2), (1, [5, 6], 4), (2, [3, 4], 2)])
def test_report_from_device_plan(cfg, problems, K, gpu):
    w = W.WORKLOADS[cfg]
    print(f"[report] workload {cfg} problems {problems} K={K}", flush=True)
    ids, L = oracle_inputs(w, problems)
    C = W.cost_matrix(w)
    ref_plan, T32 = _oracle_plan(w, ids, L, C, K)
    Bp, Ba = taot.topology_pref(C)
    home_np = W.home_map(w)
    home = torch.from_numpy(home_np).to(gpu)
    loads = taot.plan_loads(torch.from_numpy(ids).to(gpu), home, w.E)
    flow = taot.sinkhorn_batched(loads.supply, loads.demand, torch.from_numpy(C).to(gpu), w.eps, w.iters)
    sched = taot.round_schedule(loads.n, loads.spill, loads.spare, loads.excess, loads.alpha, home,
                                torch.from_numpy(T32).to(gpu), torch.from_numpy(Bp).to(gpu),
                                torch.from_numpy(Ba).to(gpu), K, w.price_step, 0)
    torch.cuda.synchronize()
    dev_plan = taot.Plan(loads, flow, sched)
    idx = list(range(len(problems)))
    got = taot.plan_report(dev_plan, home, K, problems=idx)
    want = taot.plan_report(ref_plan, torch.from_numpy(home_np), K, problems=idx)
    assert got.splitlines() == want.splitlines()
    assert got.count("== plan report") == len(problems)
    assert got.count("-> slot") == int((ref_plan.schedule.slot_expert >= 0).sum())
