"""The other full batches in the launch configuration the benchmark times:
the R = 64 (58 problems), R = 128 (384 problems) and R = 1024 (64 problems,
2^26 routing ids each) workloads, one plan_loads, one sinkhorn_batched and
one round_schedule call over the whole batch from device-generated ids.

Sampled problems are compared with the oracle, recomputed one by one from
host-generated ids: histogram and marginals bit-exact, the plan within
relative L1 1e-4, and the schedule bit-exact when the batch is scheduled
again with the sampled problems' plans replaced by the oracle's (cast to
fp32).  Every problem of the batch is checked for status, finiteness,
support and column error."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2608_03676_amd as taot
import workloads as W
from helpers import sinkhorn_check

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cfg,sample", [(1, [0, 29, 57]), (2, [0, 191, 383]), (4, [63])])
def test_full_batch(cfg, sample, gpu):
    w = W.WORKLOADS[cfg]
    B, R, E, K = w.B, w.R, w.E, w.K
    print(f"[fullsize] workload {cfg}: B={B} R={R} E={E} N={w.N}, sample {sample}", flush=True)
    home_np, C_np = W.home_map(w), W.cost_matrix(w)
    Bp_np, Ba_np = taot.topology_pref(C_np)
    home, C, Bp, Ba = (torch.from_numpy(x).to(gpu) for x in (home_np, C_np, Bp_np, Ba_np))
    ids = W.workload_ids_device(w, gpu)
    L = taot.plan_loads(ids, home, E)
    F = taot.sinkhorn_batched(L.supply, L.demand, C, w.eps, w.iters)
    S_ = taot.round_schedule(L.n, L.spill, L.spare, L.excess, L.alpha, home, F.T, Bp, Ba, K, w.price_step, 0)
    torch.cuda.synchronize()
    del ids
    torch.cuda.empty_cache()

    # every problem
    assert torch.all(L.status == 0) and torch.all(L.bad_ids == 0)
    assert torch.all(L.n.sum(dim=2, dtype=torch.int64) == w.N)
    assert torch.all(F.status == 0)
    assert bool(torch.isfinite(F.T).all()) and bool((F.T >= 0).all())
    off = ~((L.excess > 0)[:, :, None] & (L.spare > 0)[:, None, :])
    assert float(F.T.masked_select(off).abs().max()) == 0.0
    b = L.demand.double()
    mass = torch.minimum(L.supply.double().sum(1), b.sum(1))
    col = (F.T.double().sum(1) - b).abs().sum(1)
    assert bool((col <= 1e-5 * mass).all()), float((col / mass).max())
    assert torch.all(S_.unfilled == 0)
    print(f"[fullsize] workload {cfg}: batch checked", flush=True)

    # sampled problems against the oracle
    idx = torch.tensor(sample, device=gpu)
    ref = O.plan_loads(np.stack([W.problem_ids_host(w, p) for p in sample]), home_np, E)
    for name, rname in (("n", "n"), ("load_e", "x"), ("load_r", "load"), ("excess", "excess"), ("spare", "spare"),
                        ("spill", "spill")):
        assert np.array_equal(getattr(L, name).index_select(0, idx).cpu().numpy(), getattr(ref, rname)), name
    for name in ("rho", "alpha"):
        assert getattr(L, name).index_select(0, idx).cpu().numpy().tobytes() == getattr(ref, name).tobytes(), name
    a, d = ref.excess.astype(float), ref.spare.astype(float)
    plan = O.sinkhorn(a, d, C_np.astype(float), w.eps, w.iters)
    sinkhorn_check(F.T.index_select(0, idx).cpu().numpy(), plan.T, a, d)
    print(f"[fullsize] workload {cfg}: loads and plans of the sample match", flush=True)

    T32 = plan.T.astype(np.float32)
    Tmix = F.T.clone()
    Tmix.index_copy_(0, idx, torch.from_numpy(T32).to(gpu))
    s = taot.round_schedule(L.n, L.spill, L.spare, L.excess, L.alpha, home, Tmix, Bp, Ba, K, w.price_step, 0)
    torch.cuda.synchronize()
    del Tmix
    se, sa, used = O.phase2(ref.spill, ref.spare, ref.excess, ref.alpha, home_np, T32, Bp_np, K)
    X, unfilled, rounds, status = O.phase3(ref.n, se, sa, Ba_np, K, w.price_step)
    assert np.array_equal(s.slot_expert.index_select(0, idx).cpu().numpy(), se)
    assert np.array_equal(s.slot_amount.index_select(0, idx).cpu().numpy(), sa)
    assert np.array_equal(s.X.index_select(0, idx).cpu().numpy(), X)
    assert np.array_equal(s.unfilled.index_select(0, idx).cpu().numpy(), unfilled)
    ru = s.rounds_used.index_select(0, idx).cpu().numpy()
    assert np.array_equal(ru[:, 0], used) and np.array_equal(ru[:, 1], rounds)
    torch.cuda.empty_cache()
