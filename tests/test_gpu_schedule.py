"""GPU parity of taot_round_schedule (Phase 2 + Phase 3) with the oracle:
bit-exact when both sides consume the same fp32 plan (the oracle's plan cast
to fp32)."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2608_03676_amd as taot
import workloads as W
from helpers import oracle_inputs

pytestmark = pytest.mark.gpu


def _to(x, dt=None):
    return torch.from_numpy(np.ascontiguousarray(x if dt is None else x.astype(dt))).to("cuda:0")


def _compare(L, home, T32, Bp, Ba, K, t_max=0, eta=2.0 ** -6, label="", flags=0):
    se, sa, used = O.phase2(L.spill, L.spare, L.excess, L.alpha, home, T32, Bp, K, flags=flags)
    X, unfilled, rounds, status = O.phase3(L.n, se, sa, Ba, K, eta, t_max)
    s = taot.round_schedule(_to(L.n), _to(L.spill), _to(L.spare), _to(L.excess), _to(L.alpha),
                            _to(home, np.int32), _to(T32), _to(Bp), _to(Ba), K, eta, t_max, flags=flags)
    torch.cuda.synchronize()
    assert np.array_equal(s.slot_expert.cpu().numpy(), se), f"{label} slot experts"
    assert np.array_equal(s.slot_amount.cpu().numpy(), sa), f"{label} slot amounts"
    assert np.array_equal(s.X.cpu().numpy(), X), f"{label} token split"
    assert np.array_equal(s.unfilled.cpu().numpy(), unfilled), f"{label} unfilled"
    ru = s.rounds_used.cpu().numpy()
    assert np.array_equal(ru[:, 0], used), f"{label} phase-2 iterations"
    assert np.array_equal(ru[:, 1], rounds), f"{label} phase-3 rounds"
    assert np.array_equal(s.status.cpu().numpy().view(np.uint32), status), f"{label} status"
    return se, sa, X, unfilled


@pytest.mark.parametrize("cfg,problems", [(0, [0]), (1, list(range(0, 58, 4))), (2, [0, 100, 383]),
                                          (3, [0, 1951])])
@pytest.mark.parametrize("K", [2, 4])
def test_workloads(cfg, problems, K, gpu):
    w = W.WORKLOADS[cfg]
    print(f"[schedule parity] workload {cfg} problems {problems} K={K}", flush=True)
    _, L = oracle_inputs(w, problems)
    C = W.cost_matrix(w)
    P = O.sinkhorn(L.excess.astype(float), L.spare.astype(float), C.astype(float), w.eps, w.iters)
    Bp, Ba = O.topology_pref(C)
    se, sa, X, unfilled = _compare(L, W.home_map(w), P.T.astype(np.float32), Bp, Ba, K, label=f"cfg{cfg}")
    assert np.all(unfilled == 0)


@pytest.mark.parametrize("flags", [taot.SCH_NO_TOPO, taot.SCH_NO_FLOW, taot.SCH_NO_TOPO | taot.SCH_NO_FLOW,
                                   taot.SCH_ROW_PRIORITY, taot.SCH_ROW_PRIORITY | taot.SCH_NO_TOPO])
@pytest.mark.parametrize("cfg,problems", [(1, list(range(0, 58, 8))), (3, [0, 977])])
def test_score_ablations(cfg, problems, flags, gpu):
    """The Phase-2 ablations (score terms dropped, row-priority matching),
    bit-exact against the oracle with the same flags."""
    w = W.WORKLOADS[cfg]
    print(f"[schedule parity] workload {cfg} problems {problems} flags {flags}", flush=True)
    _, L = oracle_inputs(w, problems)
    C = W.cost_matrix(w)
    P = O.sinkhorn(L.excess.astype(float), L.spare.astype(float), C.astype(float), w.eps, w.iters)
    Bp, Ba = O.topology_pref(C)
    _compare(L, W.home_map(w), P.T.astype(np.float32), Bp, Ba, w.K, label=f"cfg{cfg} flags {flags}",
             flags=flags)


def _random_instance(seed):
    rng = np.random.default_rng(seed)
    R = int(rng.integers(2, 40))
    E = int(rng.integers(1, 4 * R + 1))
    N = int(rng.integers(10, 300))
    B = 3
    p = rng.dirichlet(np.full(E, 0.4))
    ids = rng.choice(E, size=(B, R, N), p=p).astype(np.int32)
    home = rng.integers(0, R, size=E).astype(np.int32)
    L = O.plan_loads(ids, home, E)
    C = W.cost_matrix_for(R, ("three_tier", 1.0, 3.0, 8.0, 16))
    P = O.sinkhorn(L.excess.astype(float), L.spare.astype(float), C.astype(float), 0.3, 40)
    Bp, Ba = O.topology_pref(C)
    return L, home, P.T.astype(np.float32), Bp, Ba


@pytest.mark.parametrize("seed", range(16))
@pytest.mark.parametrize("K", [0, 1, 3])
def test_random(seed, K, gpu):
    L, home, T32, Bp, Ba = _random_instance(seed)
    _compare(L, home, T32, Bp, Ba, K, label=f"seed{seed}")


def test_starved_auction_reports_unfilled(gpu):
    L, home, T32, Bp, Ba = _random_instance(99)
    se, sa, X, unfilled = _compare(L, home, T32, Bp, Ba, 2, t_max=2)
    assert np.any(unfilled > 0)


def test_uninformative_hint_and_negative_scores(gpu):
    """A zero plan leaves the OT term at 0; a large price step drives auction
    scores negative, exercising the ordered keys of the arbitration."""
    L, home, T32, Bp, Ba = _random_instance(7)
    _compare(L, home, np.zeros_like(T32), Bp, Ba, 2, eta=0.75)


def _instance(seed, R, E=None, N=None, B=2):
    rng = np.random.default_rng(seed)
    E = E or int(rng.integers(R, 2 * R + 1))
    N = N or int(rng.integers(50, 400))
    p = rng.dirichlet(np.full(E, 0.4))
    ids = rng.choice(E, size=(B, R, N), p=p).astype(np.int32)
    home = rng.integers(0, R, size=E).astype(np.int32)
    L = O.plan_loads(ids, home, E)
    C = W.cost_matrix_for(R, ("three_tier", 1.0, 3.0, 8.0, 32))
    P = O.sinkhorn(L.excess.astype(float), L.spare.astype(float), C.astype(float), 0.3, 40)
    Bp, Ba = O.topology_pref(C)
    return rng, L, home, P.T.astype(np.float32), Bp, Ba


@pytest.mark.parametrize("R", [63, 64, 65, 130, 200, 256, 300])
def test_rank_counts(R, gpu):
    """Rank sets span one to five 64-bit words (ragged last word).  With E in
    [R, 2R] some instances hold more distinct slot experts than the LDS layout
    and run on the general kernel."""
    print(f"[schedule parity] R={R}", flush=True)
    _, L, home, T32, Bp, Ba = _instance(300 + R, R)
    _compare(L, home, T32, Bp, Ba, 2, label=f"R{R}")


@pytest.mark.parametrize("eta", [0.0, 2.0 ** -6, 0.5, 1e-300, -0.25])
def test_price_steps(eta, gpu):
    """Step 0 keeps every price at 0 (lowest rank of the best tier); a step
    below the spacing of doubles makes prices stall, so service counts no
    longer order the scores and the general kernel takes over, as it does
    for a negative step."""
    _, L, home, T32, Bp, Ba = _instance(77, 96)
    _compare(L, home, T32, Bp, Ba, 2, eta=eta, label=f"eta{eta}")


@pytest.mark.parametrize("kind", ["few", "few_neg_inf", "many", "pos_inf", "five"])
def test_bonus_structures(kind, gpu):
    """Auction bonuses other than topology tiers: few distinct values per
    column (random, with -inf and NaN entries that can never win), more values than
    the tier search keeps, and +inf bonuses (both sent to the general kernel)."""
    rng, L, home, T32, Bp, _ = _instance(11, 80)
    R = 80
    if kind.startswith("few") or kind == "five":
        pool = np.array([1.5, 0.75, 0.0, -0.25, -2.0, 3.0])
        nv = 5 if kind == "five" else 4
        Ba = np.empty((R, R))
        for h in range(R):
            vals = rng.choice(pool, size=nv, replace=False)
            Ba[:, h] = vals[rng.integers(0, nv, size=R)]
        if kind == "few_neg_inf":
            Ba[rng.random((R, R)) < 0.1] = -np.inf
            Ba[rng.random((R, R)) < 0.05] = np.nan
    elif kind == "many":
        Ba = rng.uniform(-1.0, 1.0, (R, R))
    else:
        Ba = O.topology_pref(W.cost_matrix_for(R, ("two_tier", 1.0, 4.0)))[1]
        Ba[3, :] = np.inf
    _compare(L, home, T32, Bp, Ba, 2, label=kind)


@pytest.mark.parametrize("R", [300, 512, 777, 1024])
def test_large_rank_counts(R, gpu):
    """R > 256 with few experts: the 1024-thread LDS layout (rank sets of up
    to 16 words, fat-tree tiers aligned and unaligned to 64-rank words)."""
    print(f"[schedule parity] large R={R}", flush=True)
    rng = np.random.default_rng(900 + R)
    E, N, B = 96, 200, 2
    p = rng.dirichlet(np.full(E, 0.4))
    ids = rng.choice(E, size=(B, R, N), p=p).astype(np.int32)
    home = rng.integers(0, R, size=E).astype(np.int32)
    L = O.plan_loads(ids, home, E)
    C = W.cost_matrix_for(R, ("fat_tree", 1.0, 4.0, 16.0, 64) if R % 2 == 0 else ("three_tier", 1.0, 3.0, 8.0, 40))
    P = O.sinkhorn(L.excess.astype(float), L.spare.astype(float), C.astype(float), 0.3, 40)
    Bp, Ba = O.topology_pref(C)
    _compare(L, home, P.T.astype(np.float32), Bp, Ba, 2, label=f"R{R}")


@pytest.mark.parametrize("t_max", [0, 5])
def test_bid_groups(t_max, gpu):
    """The 1024-thread layout with few experts and three distinct bonus
    columns: slots of one (bonus column, expert) group bid alike, only the
    lowest open one is listed, and the next takes over when it fills (many
    such hand-overs here); with a round cap, slots still waiting count as
    unfilled."""
    R, K, E, N, B = 512, 2, 8, 400, 2
    print(f"[schedule parity] bid groups R={R} t_max={t_max}", flush=True)
    rng = np.random.default_rng(4242)
    p = rng.dirichlet(np.full(E, 0.3))
    ids = rng.choice(E, size=(B, R, N), p=p).astype(np.int32)
    home = rng.integers(0, R, size=E).astype(np.int32)
    L = O.plan_loads(ids, home, E)
    C = W.cost_matrix_for(R, ("fat_tree", 1.0, 4.0, 16.0, 64))
    P = O.sinkhorn(L.excess.astype(float), L.spare.astype(float), C.astype(float), 0.3, 40)
    Bp, _ = O.topology_pref(C)
    pool = np.array([1.5, 0.75, 0.0, -0.25])
    cols = [pool[rng.integers(0, 4, size=R)] for _ in range(3)]
    Ba = np.stack([cols[h % 3] for h in range(R)], axis=1)
    se, sa, X, unfilled = _compare(L, home, P.T.astype(np.float32), Bp, Ba, K, t_max=t_max, label=f"groups t{t_max}")
    # the instance really has large groups
    open_ = (se >= 0) & (sa > 0)
    keys = {(b, h % 3, e) for b in range(B) for h, e in zip(np.nonzero(open_[b])[0] // K, se[b][open_[b]])}
    assert open_.sum() >= 4 * len(keys)


def test_workload4_problem(gpu):
    """One problem of the R = 1024 workload (4096 experts, ~11000 auction rounds)."""
    w = W.WORKLOADS[4]
    print("[schedule parity] workload 4 problem 0", flush=True)
    _, L = oracle_inputs(w, [0])
    C = W.cost_matrix(w)
    P = O.sinkhorn(L.excess.astype(float), L.spare.astype(float), C.astype(float), w.eps, w.iters)
    Bp, Ba = O.topology_pref(C)
    _compare(L, W.home_map(w), P.T.astype(np.float32), Bp, Ba, w.K, label="cfg4")


@pytest.mark.parametrize("R,K", [(16, 2), (48, 4), (100, 2), (200, 2)])
def test_large_batches(R, K, gpu):
    """Batches of more than six problems per compute unit take the
    register-capped builds of the LDS kernels (eight problems per compute
    unit): the one-wave configuration up to R = 64, the 256-thread one
    above, which packs its auction list (one slot per thread at R K <= 256,
    two above); every problem bit-exact with the oracle."""
    B = 1600 if R <= 64 else 1700
    print(f"[schedule parity] large batch B={B} R={R} K={K}", flush=True)
    _, L, home, T32, Bp, Ba = _instance(500 + R, R, E=2 * R, N=120, B=B)
    _compare(L, home, T32, Bp, Ba, K, label=f"B{B} R{R}")
