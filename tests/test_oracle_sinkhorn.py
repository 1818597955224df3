"""Pins of the oracle's Phase-1 Sinkhorn (Sec. A.2) against closed forms,
brute-force optimal transport, a library LP solver and invariants."""
import itertools
import math

import numpy as np
import pytest
from scipy.optimize import linprog

import oracle as O
import workloads as W


def _marg(R, rng, lo=1, hi=50):
    """Integer supply/demand with equal mass on disjoint supports."""
    a = np.zeros(R)
    b = np.zeros(R)
    hot = rng.choice(R, size=max(1, R // 3), replace=False)
    cold = np.setdiff1d(np.arange(R), hot)
    a[hot] = rng.integers(lo, hi, size=hot.size)
    b[cold] = rng.multinomial(int(a.sum()), np.full(cold.size, 1.0 / cold.size))
    return a, b


def test_zero_cost_gives_outer_product():
    """C = 0: after one iteration T = a b^T / mass in exact arithmetic
    (u = a/R, v = b R/mass); the log-domain exp/log round trips leave ~1e-13."""
    rng = np.random.default_rng(1)
    for R in (3, 8, 17):
        a, b = _marg(R, rng)
        mass = a.sum()
        for iters in (1, 2, 7):
            P = O.sinkhorn(a, b, np.zeros((R, R)), eps=0.37, iters=iters)
            np.testing.assert_allclose(P.T[0], np.outer(a, b) / mass, rtol=1e-12, atol=0)


@pytest.mark.parametrize("scale", [1e3, 1e6])
def test_large_eps_approaches_outer_product(scale):
    """M_ij in [exp(-Cmax/eps), 1] bounds the converged T_ij / (a_i b_j / mass)
    within [exp(-2 Cmax/eps), exp(2 Cmax/eps)]."""
    rng = np.random.default_rng(2)
    R = 12
    C = W.cost_matrix_for(R, ("two_tier", 1.0, 4.0)).astype(np.float64)
    a, b = _marg(R, rng)
    eps = scale * C.max()
    P = O.sinkhorn(a, b, C, eps=eps, iters=100000, tol=1e-13)
    ref = np.outer(a, b) / a.sum()
    m = ref > 0
    ratio = P.T[0][m] / ref[m]
    lo, hi = math.exp(-2 * C.max() / eps), math.exp(2 * C.max() / eps)
    assert np.all(ratio >= lo * (1 - 1e-12)) and np.all(ratio <= hi * (1 + 1e-12))
    assert np.all(P.T[0][~m] == 0)


@pytest.mark.parametrize("cfg", [0, 1])
def test_marginals_to_1e12_run_to_tolerance(cfg):
    """Run to tolerance: row and column sums hold to 1e-12 of the mass."""
    w = W.WORKLOADS[cfg]
    rng = np.random.default_rng(3 + cfg)
    R = min(w.R, 32)
    C = W.cost_matrix_for(R, w.cost).astype(np.float64)
    a, b = _marg(R, rng, 1, 1000)
    mass = a.sum()
    P = O.sinkhorn(a, b, C, eps=w.eps, iters=1_000_000, tol=1e-13, colcap=False)
    T = P.T[0]
    assert P.used[0] < 1_000_000
    assert np.abs(T.sum(1) - a).sum() <= 1e-12 * mass
    assert np.abs(T.sum(0) - b).sum() <= 1e-12 * mass


def test_fixed_n_columns_exact():
    """One iteration ends with the column update, so column sums equal the demand
    to rounding at any fixed N, while rows carry the residual."""
    w = W.WORKLOADS[2]
    rng = np.random.default_rng(4)
    R = 32
    C = W.cost_matrix_for(R, w.cost).astype(np.float64)
    a, b = _marg(R, rng, 1, 500)
    for iters in (1, 3, 10):
        T = O.sinkhorn(a, b, C, eps=w.eps, iters=iters, colcap=False).T[0]
        np.testing.assert_allclose(T.sum(0), b, rtol=1e-13, atol=1e-9)


def _integer_plans(a, b):
    """All non-negative integer matrices with row sums a and column sums b."""
    a = [int(v) for v in a]
    b = [int(v) for v in b]
    n, m = len(a), len(b)

    def rows(i, cap):
        if i == n:
            if all(c == 0 for c in cap):
                yield []
            return
        for comp in _compositions(a[i], cap):
            yield from ([list(comp)] + rest for rest in rows(i + 1, [c - x for c, x in zip(cap, comp)]))

    yield from rows(0, b)


def _compositions(total, cap):
    if len(cap) == 1:
        if total <= cap[0]:
            yield (total,)
        return
    for x in range(min(total, cap[0]) + 1):
        for rest in _compositions(total - x, cap[1:]):
            yield (x,) + rest


@pytest.mark.parametrize("seed", range(5))
def test_eps_to_zero_matches_bruteforce_ot(seed):
    """4x4, integer marginals (mass <= 10): the transportation polytope is
    totally unimodular, so the LP optimum OT* is attained by an integer plan and
    brute force finds it.  The entropic plan satisfies
    0 <= <T_eps, C> - OT* <= eps * mass * log(16) (entropy of a mass-m plan on
    16 cells lies in [-m log m, m log 16 - m log m]).  T_eps is a convex
    combination of integral vertices; if every other integer plan costs at least
    OT* + delta, the weight off the optimum is at most gap/delta, hence
    ||T_eps - X*||_1 <= 2 * mass * gap / delta."""
    rng = np.random.default_rng(10 + seed)
    R = 4
    a = rng.multinomial(int(rng.integers(4, 11)), np.full(R, 0.25)).astype(float)
    b = rng.multinomial(int(a.sum()), np.full(R, 0.25)).astype(float)
    C = rng.uniform(0.5, 4.0, size=(R, R))
    mass = a.sum()
    plans = [np.array(p, float) for p in _integer_plans(a, b)]
    costs = np.array([(p * C).sum() for p in plans])
    order = np.argsort(costs)
    best, best_plan = float(costs[order[0]]), plans[order[0]]
    delta = float(costs[order[1]] - best) if len(plans) > 1 else math.inf
    # library cross-check of OT*
    A_eq = np.zeros((2 * R, R * R))
    for i in range(R):
        A_eq[i, i * R:(i + 1) * R] = 1
        A_eq[R + i, i::R] = 1
    lp = linprog(C.ravel(), A_eq=A_eq, b_eq=np.concatenate([a, b]), bounds=(0, None), method="highs")
    assert abs(lp.fun - best) <= 1e-9 * max(1.0, best)
    gaps = []
    for frac in (1.0, 0.3, 0.1, 0.03, 0.01):
        eps = frac * C.max()
        P = O.sinkhorn(a, b, C, eps=eps, iters=2_000_000, tol=1e-12, colcap=False)
        T = P.T[0]
        gap = float((T * C).sum()) - best
        assert -1e-8 * mass <= gap <= eps * mass * math.log(R * R) + 1e-8
        if delta > 0:
            assert np.abs(T - best_plan).sum() <= 2 * mass * max(gap, 0.0) / delta + 1e-7
        gaps.append(gap)
    assert gaps[-1] <= gaps[0] + 1e-12


def test_two_by_two_closed_form():
    """Converged 2x2 plan: T = [[t, a1-t], [b1-t, a2-b1+t]] with the Gibbs cross
    ratio T11 T22 / (T12 T21) = exp(-(C11 + C22 - C12 - C21)/eps), a quadratic in t."""
    a = np.array([3.0, 5.0])
    b = np.array([2.0, 6.0])
    C = np.array([[0.3, 1.7], [2.2, 0.4]])
    eps = 0.9
    k = math.exp(-(C[0, 0] + C[1, 1] - C[0, 1] - C[1, 0]) / eps)
    # t (a2 - b1 + t) = k (a1 - t)(b1 - t)  ->  (1-k) t^2 + (a2 - b1 + k(a1+b1)) t - k a1 b1 = 0
    qa, qb, qc = 1 - k, a[1] - b[0] + k * (a[0] + b[0]), -k * a[0] * b[0]
    t = (-qb + math.sqrt(qb * qb - 4 * qa * qc)) / (2 * qa)
    ref = np.array([[t, a[0] - t], [b[0] - t, a[1] - b[0] + t]])
    P = O.sinkhorn(a, b, C, eps=eps, iters=100000, tol=1e-15, colcap=False)
    np.testing.assert_allclose(P.T[0], ref, rtol=1e-12)


def test_gibbs_cross_ratio_any_iteration():
    """T = diag(u) M diag(v): T_ij T_kl / (T_il T_kj) = M_ij M_kl / (M_il M_kj)
    at every iteration count."""
    rng = np.random.default_rng(5)
    R = 6
    a = rng.uniform(1, 5, R)
    b = rng.uniform(1, 5, R)
    b *= a.sum() / b.sum()
    C = rng.uniform(0, 3, (R, R))
    eps = 0.7
    for iters in (1, 4, 40):
        T = O.sinkhorn(a, b, C, eps=eps, iters=iters, colcap=False).T[0]
        for (i, k), (j, l) in itertools.product(itertools.combinations(range(R), 2), repeat=2):
            if j == l:
                continue
            lhs = T[i, j] * T[k, l] / (T[i, l] * T[k, j])
            rhs = math.exp(-(C[i, j] + C[k, l] - C[i, l] - C[k, j]) / eps)
            assert abs(lhs / rhs - 1) < 1e-12


def test_intra_inter_kernel_ratio_eps_lambda():
    """With eps = lambda and W = 1 intra / lambda inter, M_intra / M_inter =
    exp((lambda - 1)/lambda): check it on the plan of a supply row facing two
    equally demanding columns, one intra- and one inter-node."""
    lam = 3.0
    C = np.array([[0.0, 1.0, lam], [1.0, 0.0, lam], [lam, lam, 0.0]])
    a = np.array([4.0, 0.0, 0.0])
    b = np.array([0.0, 2.0, 2.0])
    P = O.sinkhorn(a, b, C, eps=lam, iters=1, colcap=False)
    T = P.T[0]
    u0 = math.exp(P.f[0][0] / lam)
    g1, g2 = P.g[0][1], P.g[0][2]
    M01 = T[0, 1] / (u0 * math.exp(g1 / lam))
    M02 = T[0, 2] / (u0 * math.exp(g2 / lam))
    assert abs(M01 / M02 - math.exp((lam - 1) / lam)) < 1e-12


def test_invariances():
    rng = np.random.default_rng(6)
    R = 10
    C = rng.uniform(0.5, 3.0, (R, R))
    np.fill_diagonal(C, 0)
    a, b = _marg(R, rng)
    eps = 0.4
    base = O.sinkhorn(a, b, C, eps=eps, iters=30).T[0]
    # adding a constant to each row of C leaves every iterate unchanged
    rowc = rng.uniform(-2, 2, R)[:, None]
    np.testing.assert_allclose(O.sinkhorn(a, b, C + rowc, eps=eps, iters=30).T[0], base, rtol=1e-10, atol=1e-12)
    # scaling both marginals by c scales the plan by c
    np.testing.assert_allclose(O.sinkhorn(3 * a, 3 * b, C, eps=eps, iters=30).T[0], 3 * base, rtol=1e-11, atol=1e-12)
    # a joint permutation of ranks permutes the plan
    p = rng.permutation(R)
    Tp = O.sinkhorn(a[p], b[p], C[np.ix_(p, p)], eps=eps, iters=30).T[0]
    np.testing.assert_allclose(Tp, base[np.ix_(p, p)], rtol=1e-11, atol=1e-12)
    # column constants leave the converged plan unchanged
    colc = rng.uniform(-2, 2, R)[None, :]
    T1 = O.sinkhorn(a, b, C, eps=eps, iters=10**6, tol=1e-14).T[0]
    T2 = O.sinkhorn(a, b, C + colc, eps=eps, iters=10**6, tol=1e-14).T[0]
    np.testing.assert_allclose(T2, T1, rtol=1e-9, atol=1e-10)


@pytest.mark.parametrize("cfg", [0, 1])
def test_log_and_linear_domains_agree(cfg):
    """The log-domain oracle and the literal linear-domain GEMV form agree where
    M = exp(-C/eps) stays far above underflow."""
    w = W.WORKLOADS[cfg]
    R = min(w.R, 24)
    C = W.cost_matrix_for(R, w.cost).astype(np.float64)
    rng = np.random.default_rng(7)
    a, b = _marg(R, rng)
    assert math.exp(-C.max() / w.eps) > 1e-300
    Pl = O.sinkhorn(a, b, C, eps=w.eps, iters=w.iters, domain="log")
    Pn = O.sinkhorn(a, b, C, eps=w.eps, iters=w.iters, domain="linear")
    np.testing.assert_allclose(Pl.T[0], Pn.T[0], rtol=1e-9, atol=1e-9 * a.sum())


def test_zero_mass_and_bad_input():
    R = 4
    C = np.ones((R, R))
    P = O.sinkhorn(np.zeros(R), np.ones(R), C, eps=1.0, iters=3)
    assert P.status[0] == O.ST_ZERO_MASS and not P.T.any() and np.all(np.isneginf(P.f))
    a = np.array([1.0, np.nan, 0, 0])
    P = O.sinkhorn(a, np.ones(R), C, eps=1.0, iters=3)
    assert P.status[0] == O.ST_BAD_INPUT and not P.T.any()
    Cb = C.copy()
    Cb[1, 2] = np.inf
    P = O.sinkhorn(np.array([1.0, 0, 0, 0]), np.array([0, 1.0, 0, 0]), Cb, eps=1.0, iters=3)
    assert P.status[0] == O.ST_BAD_INPUT
    with pytest.raises(ValueError):
        O.sinkhorn(np.ones(R), np.ones(R), C, eps=0.0, iters=3)
    with pytest.raises(ValueError):
        O.sinkhorn(np.ones(R), np.ones(R), C, eps=1.0, iters=0)


def test_supply_scaling_and_column_cap():
    """gamma = min(1, sum d / sum s) rescales an oversized supply, and the column
    cap keeps every column at or below its demand."""
    R = 5
    C = W.cost_matrix_for(R, ("two_tier", 1.0, 4.0)).astype(np.float64)
    a = np.array([7.0, 5.0, 0, 0, 0])
    b = np.array([0, 0, 4.0, 3.0, 2.0])
    P = O.sinkhorn(a, b, C, eps=0.2, iters=50)
    T = P.T[0]
    assert np.all(T.sum(0) <= b * (1 + 1e-15))
    np.testing.assert_allclose(T.sum(), b.sum(), rtol=1e-9)
    # rows sum to gamma * a with gamma = 9/12
    np.testing.assert_allclose(T.sum(1), a * 9.0 / 12.0, rtol=1e-6)


def test_column_cap_where_it_binds():
    """The cap step alone (Sec. A.2) on hand-made plans whose columns exceed
    their demand: such a column is scaled down to d_j / (c_j + eps0) of
    itself; a column at or below its demand, or empty, is left as it is
    (the factor is capped at 1, never scaled up); rows are not touched."""
    T = np.array([[2.0, 1.0, 0.0, 3.0],
                  [2.0, 1.0, 0.0, 1.0],
                  [4.0, 0.0, 0.0, 0.0]])
    T4 = np.zeros((4, 4))
    T4[:3] = T
    b = np.array([2.0, 5.0, 1.0, 4.0])   # column sums 8, 2, 0, 4
    out = O.column_cap(T4, b)[0]
    f0 = 2.0 / (8.0 + O.EPS0)             # binds: 8 -> 2
    f3 = min(1.0, 4.0 / (4.0 + O.EPS0))   # at its demand: 1 - 2.5e-13
    expect = T4.copy()
    expect[:, 0] *= f0
    expect[:, 3] *= f3
    np.testing.assert_array_equal(out, expect)
    np.testing.assert_allclose(out.sum(0), [2.0, 2.0, 0.0, 4.0], rtol=1e-12)
    assert out[0, 1] == 1.0 and out[1, 1] == 1.0  # under its demand: not scaled up


def test_column_cap_applies_once_to_the_final_plan():
    """sinkhorn(colcap) equals the cap step applied to sinkhorn(no colcap),
    bit for bit: the cap runs once, after the last iteration, on the final
    plan (reading R8), at several iteration counts and with gamma < 1."""
    rng = np.random.default_rng(5)
    R = 9
    C = rng.uniform(0.0, 3.0, (R, R))
    a = np.zeros((2, R))
    b = np.zeros((2, R))
    a[0, :3], b[0, 3:] = rng.integers(1, 40, 3), rng.integers(1, 40, 6)
    a[1, :4], b[1, 4:] = rng.integers(30, 90, 4), rng.integers(1, 20, 5)  # supply above demand
    for iters in (1, 2, 7, 40):
        P1 = O.sinkhorn(a, b, C, eps=0.3, iters=iters, colcap=True)
        P0 = O.sinkhorn(a, b, C, eps=0.3, iters=iters, colcap=False)
        assert P1.T.tobytes() == O.column_cap(P0.T, b).tobytes()
        assert np.all(P1.T.sum(1) <= P0.T.sum(1) * (1 + 1e-15))


@pytest.mark.parametrize("eps,gamma", [(3.0, 1.0), (0.08, 1.0), (3.0, 0.8)])
def test_single_overloaded_rank(eps, gamma):
    """One supply row (one overloaded rank, as in the hot-rank workloads of
    Sec. 4.4): the column marginals alone fix the plan, T[h] = d, whatever
    the costs and eps; with supply above demand gamma scales it back."""
    rng = np.random.default_rng(11)
    R = 16
    C = W.cost_matrix_for(R, ("two_tier", 1.0, 3.0)).astype(np.float64)
    h = 5
    b = rng.integers(1, 900, size=R).astype(float)
    b[h] = 0
    a = np.zeros(R)
    a[h] = b.sum() / gamma
    P = O.sinkhorn(a, b, C, eps=eps, iters=3)
    T = P.T[0]
    np.testing.assert_allclose(T[h], b, rtol=1e-12, atol=0)
    assert np.all(np.delete(T, h, axis=0) == 0)
