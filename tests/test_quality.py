"""Plan-quality metrics of the binding (tensor ops, here on the CPU) against
the oracle's plain loops: post-plan loads, rho after, intra / inter replica
counts and the weighted cost, on random schedules with empty slots and a
problem without load."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2608_03676_amd as taot


@pytest.mark.parametrize("seed,R,E,K,rpn", [(0, 16, 40, 2, 4), (1, 8, 8, 1, 8), (2, 64, 256, 4, 8), (3, 5, 3, 3, 2)])
def test_plan_quality_matches_oracle(seed, R, E, K, rpn):
    rng = np.random.default_rng(seed)
    B, S = 4, R * K
    load = rng.integers(0, 1000, size=(B, R)).astype(np.int64)
    load[1] = 0  # no load: rho after is 0
    home = rng.integers(0, R, size=E).astype(np.int32)
    se = rng.integers(-1, E, size=(B, S)).astype(np.int32)
    X = rng.integers(0, 5, size=(B, R, S)).astype(np.int32)
    X[se[:, None, :].repeat(R, 1) < 0] = 0  # empty slots receive nothing
    m = O.metrics(load, home, se, X, K, ranks_per_node=rpn, w_inter=3.0)
    sch = taot.Schedule(torch.from_numpy(se), torch.zeros((B, S), dtype=torch.int64), torch.from_numpy(X),
                        torch.zeros(B, dtype=torch.int64), torch.zeros((B, 2), dtype=torch.int32),
                        torch.zeros(B, dtype=torch.int32))
    q = taot.plan_quality(torch.from_numpy(load), torch.from_numpy(home), sch, K, ranks_per_node=rpn, w_inter=3.0)
    assert np.array_equal(q.load_after.numpy(), m["load_after"])
    assert q.rho_after.numpy().tobytes() == m["rho_after"].tobytes()
    assert np.array_equal(q.intra.numpy(), m["intra"]) and np.array_equal(q.inter.numpy(), m["inter"])
    assert q.weighted.numpy().tobytes() == m["weighted"].tobytes()


def _plan_from_oracle(seed, R=16, E=40, K=2, N=400):
    """A small planner run through the oracle, wrapped in the binding's
    dataclasses as CPU tensors (the report formats whatever plan it gets)."""
    rng = np.random.default_rng(seed)
    p = rng.dirichlet(np.full(E, 0.3))
    ids = rng.choice(E, size=(2, R, N), p=p).astype(np.int32)
    home = (np.arange(E) % R).astype(np.int32)
    L = O.plan_loads(ids, home, E)
    C = np.where((np.arange(R)[:, None] // 8) == (np.arange(R)[None, :] // 8), 1.0, 4.0).astype(np.float32)
    np.fill_diagonal(C, 0.0)
    P = O.sinkhorn(L.excess.astype(float), L.spare.astype(float), C.astype(float), 0.2, 100)
    Bp, Ba = O.topology_pref(C)
    se, sa, used = O.phase2(L.spill, L.spare, L.excess, L.alpha, home, P.T.astype(np.float32), Bp, K)
    X, unfilled, rounds, st = O.phase3(L.n, se, sa, Ba, K)
    t = torch.from_numpy
    loads = taot.Loads(t(L.n), t(L.x), t(L.load), t(L.excess), t(L.spare), t(L.spill),
                       t(L.excess.astype(np.float32)), t(L.spare.astype(np.float32)), t(L.rho), t(L.alpha),
                       t(L.bad), t(L.status.view(np.int32)))
    flow = taot.Flow(t(P.T.astype(np.float32)), t(P.f.astype(np.float32)), t(P.g.astype(np.float32)),
                     torch.zeros(2, dtype=torch.int32))
    sched = taot.Schedule(t(se), t(sa), t(X), t(unfilled), torch.zeros((2, 2), dtype=torch.int32),
                          t(st.view(np.int32)))
    return taot.Plan(loads, flow, sched), home, L, se, X


def test_plan_report_parts():
    """The four parts of the report: every rank's load before and after, the
    hot ranks and experts, one line per cloned expert, and copy counts, cost
    and rho that agree with the oracle's metrics."""
    K = 2
    plan, home, L, se, X = _plan_from_oracle(4, K=K)
    m = O.metrics(L.load, home, se, X, K, ranks_per_node=8, w_inter=3.0)
    rep = taot.plan_report(plan, torch.from_numpy(home), K, problems=[1])
    assert "problem 1" in rep and "problem 0" not in rep
    for tag in ("[1] load before routing", "[2] cloning plan", "[3] projected load after routing", "[4] summary"):
        assert tag in rep
    assert rep.count("-> slot") == int((se[1] >= 0).sum())
    assert rep.count("      expert") - rep.count("-> slot") == int((L.spill[1] > 0).sum())
    assert f"{int(m['intra'][1])} intra-node, {int(m['inter'][1])} inter-node copies" in rep
    assert f"weighted cost {m['weighted'][1]:.1f}" in rep
    assert f"rho {L.rho[1]:.4f} -> {m['rho_after'][1]:.4f}" in rep
    moved = int(X[1].sum())
    assert f"rerouted {moved} of {int(L.load[1].sum())} tokens" in rep
