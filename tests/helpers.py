"""Shared helpers of the GPU parity tests (no test functions here)."""
import numpy as np

import oracle as O
import workloads as W


def oracle_inputs(w, problems):
    """Host-generated ids and the oracle's loads for a subset of a workload."""
    ids = np.stack([W.problem_ids_host(w, b) for b in problems])
    loads = O.plan_loads(ids, W.home_map(w), w.E)
    return ids, loads


def sinkhorn_check(T_gpu, T_ref, a, b, tol_rel=1e-4, tol_marg=1e-5):
    """Per-problem acceptance against the oracle plan at the same N:
    relative L1 <= tol_rel; column error sum_j |sum_i T_ij - d_j| <= tol_marg * mass;
    row error <= the oracle's own fixed-N row error + tol_marg * mass."""
    T_gpu = np.asarray(T_gpu, np.float64)
    rels = []
    for p in range(T_ref.shape[0]):
        ref, got = T_ref[p], T_gpu[p]
        gamma = min(1.0, b[p].sum() / max(a[p].sum(), 1e-12))
        s = gamma * a[p]
        mass = s.sum()
        if ref.sum() == 0:
            assert not got.any(), p
            rels.append(0.0)
            continue
        rel = np.abs(got - ref).sum() / ref.sum()
        col = np.abs(got.sum(0) - b[p]).sum()
        row_ref = np.abs(ref.sum(1) - s).sum()
        row_gpu = np.abs(got.sum(1) - s).sum()
        assert rel <= tol_rel, (p, rel)
        assert col <= tol_marg * mass, (p, col, mass)
        assert row_gpu <= row_ref + tol_marg * mass, (p, row_gpu, row_ref, mass)
        rels.append(rel)
    return rels


def potentials_check(f_gpu, g_gpu, f_ref, g_ref, eps, iters, tol_rel=1e-4):
    """Per-problem acceptance of the potentials f = eps log u, g = eps log v
    against the oracle's at the same N (both start from g = 0, so each is
    determined, not only up to a shared constant).

    * The -inf pattern (off the hot / cold sets) is equal.
    * On the support: |d f_i + d g_j| <= tol_rel eps + 2^-20 (|f_i| + |g_j|).
      f_i + g_j fixes the plan entry, T_ij = exp((f_i + g_j - C_ij) / eps),
      so this is the plan's relative tolerance per entry, plus a few fp32
      units of the potentials themselves.
    * Each potential: |d f_i|, |d g_j| <= (tol_rel + 2 iters 2^-22) eps +
      2^-20 |f|.  A shared constant (f + c, g - c) leaves the plan unchanged
      and is not damped by the iteration; each half-step may move it by the
      relative rounding of the new scalings (at most 2^-22), so after iters
      iterations it is at most 2 iters 2^-22 eps.
    Returns the largest support and per-potential deviations in units of eps."""
    f_gpu, g_gpu = np.asarray(f_gpu, np.float64), np.asarray(g_gpu, np.float64)
    worst = [0.0, 0.0]
    gauge = tol_rel + 2 * iters * 2.0 ** -22
    for p in range(f_ref.shape[0]):
        hot, cold = np.isfinite(f_ref[p]), np.isfinite(g_ref[p])
        assert np.array_equal(np.isneginf(f_ref[p]), ~hot) and np.array_equal(np.isneginf(g_ref[p]), ~cold), p
        assert np.array_equal(np.isneginf(f_gpu[p]), ~hot), (p, "f pattern")
        assert np.array_equal(np.isneginf(g_gpu[p]), ~cold), (p, "g pattern")
        if not hot.any() or not cold.any():
            continue
        fr, gr = f_ref[p][hot], g_ref[p][cold]
        df, dg = f_gpu[p][hot] - fr, g_gpu[p][cold] - gr
        dsum = np.abs(df[:, None] + dg[None, :])
        lim = tol_rel * eps + 2.0 ** -20 * (np.abs(fr)[:, None] + np.abs(gr)[None, :])
        assert np.all(dsum <= lim), (p, "f + g", float((dsum / eps).max()))
        assert np.all(np.abs(df) <= gauge * eps + 2.0 ** -20 * np.abs(fr)), (p, "f", float(np.abs(df).max() / eps))
        assert np.all(np.abs(dg) <= gauge * eps + 2.0 ** -20 * np.abs(gr)), (p, "g", float(np.abs(dg).max() / eps))
        worst[0] = max(worst[0], float((dsum / eps).max()))
        worst[1] = max(worst[1], float(max(np.abs(df).max(), np.abs(dg).max()) / eps))
    return worst


def random_loads_instance(rng, R=None, E=None, N=None):
    R = R or int(rng.integers(3, 40))
    E = E or int(rng.integers(R, 4 * R + 1))
    N = N or int(rng.integers(20, 400))
    p = rng.dirichlet(np.full(E, 0.4))
    ids = np.stack([rng.choice(E, size=N, p=p) for _ in range(R)])[None].astype(np.int32)
    home = rng.integers(0, R, size=E).astype(np.int32)
    return ids, home, E
