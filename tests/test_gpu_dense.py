"""GPU parity of the dense streamed Sinkhorn (TAOT_SK_DENSE: the log-domain
iterate over all R x R entries, no support compaction) with the fp64 oracle
at the same iteration count: the plan and potential tolerances of the other
Sinkhorn paths, shared and per-problem costs, ragged shapes across the row
blocks and LDS phases, the workload-4 shape with per-problem costs, and the
degenerate problems."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2608_03676_amd as taot
import workloads as W
from helpers import oracle_inputs, potentials_check, sinkhorn_check

pytestmark = pytest.mark.gpu


def _dense(a, b, C, eps, iters, flags=0):
    dev = torch.device("cuda:0")
    out = taot.sinkhorn_batched(torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev),
                                torch.from_numpy(np.ascontiguousarray(b, np.float32)).to(dev),
                                torch.from_numpy(np.ascontiguousarray(C, np.float32)).to(dev),
                                eps, iters, flags | taot.SK_DENSE)
    torch.cuda.synchronize()
    return (out.T.cpu().numpy(), out.f.cpu().numpy(), out.g.cpu().numpy(),
            out.status.cpu().numpy().view(np.uint32))


def _check(a32, b32, C32, eps, iters, flags=0):
    T, f, g, st = _dense(a32, b32, C32, eps, iters, flags)
    a, b = a32.astype(np.float64), b32.astype(np.float64)
    ref = O.sinkhorn(a, b, C32.astype(np.float64), eps, iters, colcap=not (flags & taot.SK_NO_COLCAP))
    ok = ref.status == 0
    assert np.all(st[ok] == taot.ST_STREAMED), st
    rels = sinkhorn_check(T[ok], ref.T[ok], a[ok], b[ok])
    worst = potentials_check(f[ok], g[ok], ref.f[ok], ref.g[ok], eps, iters)
    print(f"  max relL1 {max(rels):.2e}, potentials: max |d(f+g)| {worst[0]:.2e} eps, "
          f"max |df|, |dg| {worst[1]:.2e} eps", flush=True)
    return st, ref


@pytest.mark.parametrize("cfg,problems", [(0, [0]), (1, list(range(6))), (2, [0, 100, 383])])
def test_dense_workloads(cfg, problems, gpu):
    w = W.WORKLOADS[cfg]
    print(f"[dense parity] workload {cfg} problems {problems}", flush=True)
    _, L = oracle_inputs(w, problems)
    _check(L.excess.astype(np.float32), L.spare.astype(np.float32), W.cost_matrix(w), w.eps, w.iters)


@pytest.mark.parametrize("R", [1, 2, 5, 17, 100, 300, 1027, 1100])
@pytest.mark.parametrize("per_problem", [False, True])
def test_dense_ragged_shapes(R, per_problem, gpu):
    """R across one and several row blocks of 64, partial waves and phases,
    both row kernels (R % 4 != 0 takes the phased one: 8 columns per thread
    and 4-row phases at R = 1027) and both column-update widths (R > 1024);
    random supports with zeros on both sides; costs shared or one matrix per
    problem."""
    rng = np.random.default_rng(R * 7 + per_problem)
    B = 3
    a = np.zeros((B, R), np.float32)
    b = np.zeros((B, R), np.float32)
    for p in range(B):
        hot = rng.random(R) < 0.4
        hot[rng.integers(0, R)] = True
        a[p, hot] = rng.integers(1, 3000, size=int(hot.sum()))
        cold = ~hot if R > 1 else np.ones(R, bool)
        if not cold.any():
            cold[0] = True
        b[p, cold] = rng.integers(1, 3000, size=int(cold.sum()))
    shape = (B, R, R) if per_problem else (R, R)
    C = rng.uniform(0.0, 4.0, size=shape).astype(np.float32)
    print(f"[dense parity] R={R} per_problem={per_problem}", flush=True)
    for eps, iters, flags in ((0.5, 30, 0), (0.1, 60, 0), (0.1, 60, taot.SK_NO_COLCAP)):
        _check(a, b, C, eps, iters, flags)


def test_dense_stress_shape_per_problem_costs(gpu):
    """The workload-4 shape (R = 1024, the fat-tree costs) with one cost matrix
    per problem, fewer iterations so that the oracle stays quick."""
    w = W.WORKLOADS[4]
    problems = [0, 63]
    print(f"[dense parity] workload 4 problems {problems}, per-problem costs", flush=True)
    _, L = oracle_inputs(w, problems)
    C0 = W.cost_matrix(w)
    C = np.stack([C0 * np.float32(1.0 + 0.25 * k) for k in range(len(problems))])
    _check(L.excess.astype(np.float32), L.spare.astype(np.float32), C, w.eps, 20)


def test_dense_degenerate(gpu):
    R = 40
    rng = np.random.default_rng(3)
    a = np.zeros((4, R), np.float32)
    b = np.zeros((4, R), np.float32)
    a[1, :5] = 100.0               # no demand: zero mass
    b[2, 5:] = 10.0                # no supply
    a[3, :5] = 100.0
    b[3, 5:] = 10.0
    C = rng.uniform(0.5, 2.0, (R, R)).astype(np.float32)
    T, f, g, st = _dense(a, b, C, 0.2, 10)
    assert list(st[:3]) == [taot.ST_ZERO_MASS] * 3 and st[3] == taot.ST_STREAMED, st
    assert not T[:3].any() and np.all(np.isneginf(f[:3])) and np.all(np.isneginf(g[:3]))
    # a non-finite cost in a row the iterate never weights, and a negative supply
    Cb = np.stack([C] * 4)
    Cb[3, 30, 2] = np.nan
    a2 = a.copy()
    a2[1, 7] = -1.0
    T, f, g, st = _dense(a2, b, Cb, 0.2, 10)
    ref = O.sinkhorn(a2.astype(float), b.astype(float), Cb.astype(float), 0.2, 10)
    assert list(ref.status) == [O.ST_ZERO_MASS, O.ST_BAD_INPUT, O.ST_ZERO_MASS, O.ST_BAD_INPUT]
    assert list(st) == [taot.ST_ZERO_MASS, taot.ST_BAD_INPUT, taot.ST_ZERO_MASS, taot.ST_BAD_INPUT], st
    assert not T.any() and np.all(np.isneginf(f)) and np.all(np.isneginf(g))


def test_dense_deterministic(gpu):
    w = W.WORKLOADS[2]
    _, L = oracle_inputs(w, [1, 2])
    a, b = L.excess.astype(np.float32), L.spare.astype(np.float32)
    T1 = _dense(a, b, W.cost_matrix(w), w.eps, 100)[0]
    T2 = _dense(a, b, W.cost_matrix(w), w.eps, 100)[0]
    assert T1.tobytes() == T2.tobytes()


def test_dense_long_run_potentials_grow(gpu):
    """Enough iterations at the R = 1024 shape for the row potentials to pass
    2^7 in log2 units: the rebuilt entries of K~ in columns without demand
    must stay zero (not exp2 of a large F), so the plan stays finite and equal
    to the oracle's."""
    w = W.WORKLOADS[4]
    problems = [2, 26]
    print(f"[dense parity] workload 4 problems {problems}, 150 iterations", flush=True)
    _, L = oracle_inputs(w, problems)
    C0 = W.cost_matrix(w)
    C = np.stack([C0 * np.float32(1.0 + 0.01 * (p % 7)) for p in problems])
    T, f, g, st = _dense(L.excess.astype(np.float32), L.spare.astype(np.float32), C, w.eps, 150)
    assert np.isfinite(T).all()
    _check(L.excess.astype(np.float32), L.spare.astype(np.float32), C, w.eps, 150)


@pytest.mark.parametrize("R", [100, 1024])
def test_dense_unaligned_costs(R, gpu):
    """Costs 4 bytes off 16-byte alignment (a view into a larger buffer): the
    R % 4 == 0 shapes then take the phased row kernel instead of the
    wave-streamed one, with the same results against the oracle."""
    rng = np.random.default_rng(R + 11)
    B = 2
    a = np.zeros((B, R), np.float32)
    b = np.zeros((B, R), np.float32)
    for p in range(B):
        hot = rng.random(R) < 0.1
        hot[0] = True
        a[p, hot] = rng.integers(1, 3000, size=int(hot.sum()))
        b[p, ~hot] = rng.integers(1, 3000, size=int((~hot).sum()))
    C = rng.uniform(0.0, 4.0, size=(B, R, R)).astype(np.float32)
    dev = torch.device("cuda:0")
    flat = torch.empty(B * R * R + 1, dtype=torch.float32, device=dev)
    Cv = flat[1:].view(B, R, R)
    Cv.copy_(torch.from_numpy(C))
    assert Cv.data_ptr() % 16 == 4
    out = taot.sinkhorn_batched(torch.from_numpy(a).to(dev), torch.from_numpy(b).to(dev), Cv, 0.2, 40, taot.SK_DENSE)
    torch.cuda.synchronize()
    T, f, g = out.T.cpu().numpy(), out.f.cpu().numpy(), out.g.cpu().numpy()
    st = out.status.cpu().numpy().view(np.uint32)
    ref = O.sinkhorn(a.astype(np.float64), b.astype(np.float64), C.astype(np.float64), 0.2, 40)
    assert np.all(st == taot.ST_STREAMED), st
    sinkhorn_check(T, ref.T, a.astype(np.float64), b.astype(np.float64))
    potentials_check(f, g, ref.f, ref.g, 0.2, 40)
    # the aligned copy takes the wave-streamed kernel: the same plan to the tolerance
    T2 = _dense(a, b, C, 0.2, 40)[0]
    assert np.abs(T2.astype(np.float64) - T).sum() <= 1e-4 * np.abs(T).sum()


@pytest.mark.parametrize("cfg,problems", [(0, [0]), (1, [0, 1, 2, 3])])
def test_linear_domain_workloads(cfg, problems, gpu):
    """TAOT_SK_LINEAR (the GEMV form on M = exp(-C / eps) without
    stabilisation, Sec. A.2) against the oracle's linear-domain iterate at the
    same N, on the workloads whose M stays in fp32's normal range."""
    w = W.WORKLOADS[cfg]
    print(f"[linear parity] workload {cfg} problems {problems}", flush=True)
    _, L = oracle_inputs(w, problems)
    a32, b32, C32 = L.excess.astype(np.float32), L.spare.astype(np.float32), W.cost_matrix(w)
    T, f, g, st = _dense(a32, b32, C32, w.eps, w.iters, taot.SK_LINEAR)
    a, b = a32.astype(np.float64), b32.astype(np.float64)
    ref = O.sinkhorn(a, b, C32.astype(np.float64), w.eps, w.iters, domain="linear")
    ok = ref.status == 0
    assert np.all(st[ok] == taot.ST_STREAMED), st
    sinkhorn_check(T[ok], ref.T[ok], a[ok], b[ok])
    potentials_check(f[ok], g[ok], ref.f[ok], ref.g[ok], w.eps, w.iters)


@pytest.mark.parametrize("R", [5, 17, 100, 300])
def test_linear_domain_ragged(R, gpu):
    """The linear mode on both row kernels (odd R takes the phased one),
    costs up to 20 eps, shared and per-problem; also close to the stabilised
    dense mode, which computes the same iterate.  Supply and demand have equal
    totals, as excess and spare do: with a demand total many times the supply
    the plain scalings grow by that ratio every iteration and leave fp32's
    range within a few dozen iterations (fp64 only later), which the
    stabilised modes absorb and the linear form, by definition, does not."""
    rng = np.random.default_rng(R + 5)
    B = 3
    a = np.zeros((B, R), np.float32)
    b = np.zeros((B, R), np.float32)
    for p in range(B):
        hot = rng.random(R) < 0.3
        hot[0] = True
        hot[-1] = False
        a[p, hot] = rng.integers(1, 3000, size=int(hot.sum()))
        cold = rng.uniform(1.0, 3000.0, size=int((~hot).sum()))
        b[p, ~hot] = (cold * (a[p].sum(dtype=np.float64) / cold.sum())).astype(np.float32)
    for shape in ((R, R), (B, R, R)):
        C = rng.uniform(0.0, 2.0, size=shape).astype(np.float32)
        T, f, g, st = _dense(a, b, C, 0.1, 50, taot.SK_LINEAR)
        ref = O.sinkhorn(a.astype(np.float64), b.astype(np.float64), C.astype(np.float64), 0.1, 50, domain="linear")
        assert np.all(st == taot.ST_STREAMED), st
        sinkhorn_check(T, ref.T, a.astype(np.float64), b.astype(np.float64))
        potentials_check(f, g, ref.f, ref.g, 0.1, 50)
        Ts = _dense(a, b, C, 0.1, 50)[0]
        assert np.abs(Ts.astype(np.float64) - T).sum() <= 1e-4 * np.abs(T).sum()
