"""GPU parity on the hot-rank workloads of the paper's scalability study
(Sec. 4.4: one rank receives 30-90 % of the routing choices, EP 4-32,
K = 1-16 guest slots, eps = lambda = 3): whole batches of 48 problems in the
launch configuration the benchmark times (device-generated ids), against the
oracle on host-generated ids of every problem."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2608_03676_amd as taot
import workloads as W
from helpers import sinkhorn_check

pytestmark = pytest.mark.gpu

POINTS = [(4, 0.9, 16), (8, 0.3, 1), (16, 0.5, 2), (16, 0.7, 4), (32, 0.9, 8), (32, 0.3, 16)]


@pytest.mark.parametrize("ep,frac,K", POINTS)
def test_hot_rank_batch(ep, frac, K, gpu):
    w = W.llep_workload(ep, frac, K)
    print(f"[hot rank] EP{ep} frac {frac} K={K}: B={w.B} N={w.N}", flush=True)
    home_np, C_np = W.home_map(w), W.cost_matrix(w)
    Bp_np, Ba_np = taot.topology_pref(C_np)
    home, C, Bp, Ba = (torch.from_numpy(x).to(gpu) for x in (home_np, C_np, Bp_np, Ba_np))
    ids = W.workload_ids_device(w, gpu)
    L = taot.plan_loads(ids, home, w.E)
    F = taot.sinkhorn_batched(L.supply, L.demand, C, w.eps, w.iters)
    torch.cuda.synchronize()
    del ids

    ref = O.plan_loads(np.stack([W.problem_ids_host(w, b) for b in range(w.B)]), home_np, w.E)
    for name, rname in (("n", "n"), ("load_e", "x"), ("load_r", "load"), ("excess", "excess"), ("spare", "spare"),
                        ("spill", "spill"), ("bad_ids", "bad")):
        assert np.array_equal(getattr(L, name).cpu().numpy(), getattr(ref, rname)), name
    for name in ("rho", "alpha"):
        assert getattr(L, name).cpu().numpy().tobytes() == getattr(ref, name).tobytes(), name
    # one overloaded rank per problem: the seeded hot rank
    hot = [int(np.flatnonzero(ref.excess[b])[0]) for b in range(w.B)]
    assert all(np.count_nonzero(ref.excess[b]) == 1 for b in range(w.B))
    assert hot == [W.hot_rank(w, b) for b in range(w.B)]

    a, d = ref.excess.astype(float), ref.spare.astype(float)
    plan = O.sinkhorn(a, d, C_np.astype(float), w.eps, w.iters)
    T = F.T.cpu().numpy()
    sinkhorn_check(T, plan.T, a, d)
    for b in range(w.B):  # a single supply row: its plan row is the demand
        np.testing.assert_allclose(T[b, hot[b]], d[b], rtol=1e-5, atol=0)
        assert not np.delete(T[b], hot[b], axis=0).any()

    T32 = plan.T.astype(np.float32)
    s = taot.round_schedule(L.n, L.spill, L.spare, L.excess, L.alpha, home, torch.from_numpy(T32).to(gpu), Bp, Ba,
                            K, w.price_step, 0)
    q = taot.plan_quality(L.load_r, home, s, K, ranks_per_node=8, w_inter=3.0)
    torch.cuda.synchronize()
    se, sa, used = O.phase2(ref.spill, ref.spare, ref.excess, ref.alpha, home_np, T32, Bp_np, K)
    X, unfilled, rounds, status = O.phase3(ref.n, se, sa, Ba_np, K, w.price_step)
    assert np.array_equal(s.slot_expert.cpu().numpy(), se)
    assert np.array_equal(s.slot_amount.cpu().numpy(), sa)
    assert np.array_equal(s.X.cpu().numpy(), X)
    assert np.array_equal(s.unfilled.cpu().numpy(), unfilled)
    ru = s.rounds_used.cpu().numpy()
    assert np.array_equal(ru[:, 0], used) and np.array_equal(ru[:, 1], rounds)
    assert np.array_equal(s.status.cpu().numpy().view(np.uint32), status)
    m = O.metrics(ref.load, home_np, se, X, K, ranks_per_node=8, w_inter=3.0)
    assert q.rho_after.cpu().numpy().tobytes() == m["rho_after"].tobytes()
    assert np.array_equal(q.intra.cpu().numpy(), m["intra"]) and np.array_equal(q.inter.cpu().numpy(), m["inter"])
    if ep <= 8:  # one node: every replica stays inside it
        assert not m["inter"].any()


@pytest.mark.parametrize("ep,frac,K", [(16, 0.0, 2), (16, 1.0, 2), (8, 1.0, 16)])
def test_hot_rank_extremes(ep, frac, K, gpu):
    """frac = 0 (uniform routing: small random imbalance, several overloaded
    ranks or none) and frac = 1 (every choice on the hot rank's experts, the
    other ranks idle): loads bit-exact, plan within tolerance, schedule
    bit-exact, on a slice of the batch."""
    w = W.llep_workload(ep, frac, K)
    problems = [0, 17, 47]
    print(f"[hot rank] EP{ep} frac {frac} K={K}: problems {problems}", flush=True)
    home_np, C_np = W.home_map(w), W.cost_matrix(w)
    Bp_np, Ba_np = taot.topology_pref(C_np)
    home, C, Bp, Ba = (torch.from_numpy(x).to(gpu) for x in (home_np, C_np, Bp_np, Ba_np))
    ids = W.workload_ids_device(w, gpu, problems)
    L = taot.plan_loads(ids, home, w.E)
    F = taot.sinkhorn_batched(L.supply, L.demand, C, w.eps, w.iters)
    torch.cuda.synchronize()
    ref = O.plan_loads(np.stack([W.problem_ids_host(w, b) for b in problems]), home_np, w.E)
    for name, rname in (("n", "n"), ("excess", "excess"), ("spare", "spare"), ("spill", "spill")):
        assert np.array_equal(getattr(L, name).cpu().numpy(), getattr(ref, rname)), name
    if frac == 1.0:  # only the hot rank holds load
        for q, b in enumerate(problems):
            assert np.flatnonzero(ref.load[q]).tolist() == [W.hot_rank(w, b)]
    a, d = ref.excess.astype(float), ref.spare.astype(float)
    plan = O.sinkhorn(a, d, C_np.astype(float), w.eps, w.iters)
    sinkhorn_check(F.T.cpu().numpy(), plan.T, a, d)
    T32 = plan.T.astype(np.float32)
    s = taot.round_schedule(L.n, L.spill, L.spare, L.excess, L.alpha, home, torch.from_numpy(T32).to(gpu), Bp, Ba,
                            K, w.price_step, 0)
    torch.cuda.synchronize()
    se, sa, used = O.phase2(ref.spill, ref.spare, ref.excess, ref.alpha, home_np, T32, Bp_np, K)
    X, unfilled, rounds, status = O.phase3(ref.n, se, sa, Ba_np, K, w.price_step)
    assert np.array_equal(s.slot_expert.cpu().numpy(), se)
    assert np.array_equal(s.slot_amount.cpu().numpy(), sa)
    assert np.array_equal(s.X.cpu().numpy(), X)
    assert np.array_equal(s.unfilled.cpu().numpy(), unfilled)
