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


def random_loads_instance(rng, R=None, E=None, N=None):
    R = R or int(rng.integers(3, 40))
    E = E or int(rng.integers(R, 4 * R + 1))
    N = N or int(rng.integers(20, 400))
    p = rng.dirichlet(np.full(E, 0.4))
    ids = np.stack([rng.choice(E, size=N, p=p) for _ in range(R)])[None].astype(np.int32)
    home = rng.integers(0, R, size=E).astype(np.int32)
    return ids, home, E
