"""Pins of the oracle's histogram, loads, marginals and spill (Sec. 3.1, A.1,
A.3) against brute force, exact rational arithmetic and invariants."""
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
import workloads as W


def _random_ids(rng, B, R, N, E, bad_frac=0.0):
    ids = rng.integers(0, E, size=(B, R, N), dtype=np.int32)
    if bad_frac:
        m = rng.random(ids.shape) < bad_frac
        ids[m] = rng.choice(np.array([-1, -7, E, E + 5, 2**31 - 1, -(2**31)], dtype=np.int64),
                            size=int(m.sum())).astype(np.int32)
    return ids


@pytest.mark.parametrize("seed", range(4))
def test_histogram_matches_bincount(seed):
    rng = np.random.default_rng(seed)
    B, R, N, E = 3, 5, 257, 11
    ids = _random_ids(rng, B, R, N, E, bad_frac=0.05)
    home = rng.integers(0, R, size=E).astype(np.int32)
    L = O.plan_loads(ids, home, E)
    for b in range(B):
        nbad = 0
        for r in range(R):
            row = ids[b, r].astype(np.int64)
            ok = (row >= 0) & (row < E)
            nbad += int((~ok).sum())
            np.testing.assert_array_equal(L.n[b, r], np.bincount(row[ok], minlength=E))
        assert L.bad[b] == nbad
        assert bool(L.status[b] & O.ST_BAD_ID) == (nbad > 0)
        # invariant: sum_e n_re = N - (bad ids of rank r)
        assert L.n[b].sum() == R * N - nbad


def _brute_loads(n, home, R):
    """Independent recomputation with Python integers and Fractions."""
    E = n.shape[1]
    x = [int(n[:, e].sum()) for e in range(E)]
    load = [0] * R
    for e in range(E):
        load[int(home[e])] += x[e]
    L = sum(load)
    return x, load, L


@pytest.mark.parametrize("seed", range(6))
def test_loads_marginals_rho_alpha(seed):
    rng = np.random.default_rng(100 + seed)
    B, R, E = 2, int(rng.integers(2, 9)), int(rng.integers(2, 20))
    N = int(rng.integers(1, 300))
    ids = _random_ids(rng, B, R, N, E)
    home = rng.integers(0, R, size=E).astype(np.int32)
    L = O.plan_loads(ids, home, E)
    for b in range(B):
        x, load, Ltot = _brute_loads(L.n[b], home, R)
        np.testing.assert_array_equal(L.x[b], x)
        np.testing.assert_array_equal(L.load[b], load)
        m = Ltot // R
        assert L.mean[b] == m
        np.testing.assert_array_equal(L.excess[b], [max(v - m, 0) for v in load])
        np.testing.assert_array_equal(L.spare[b], [max(m - v, 0) for v in load])
        # sum excess - sum spare = L - R*m in [0, R-1]
        d = int(L.excess[b].sum() - L.spare[b].sum())
        assert d == Ltot - R * m and 0 <= d <= R - 1
        # hot and cold sets are disjoint
        assert not np.any((L.excess[b] > 0) & (L.spare[b] > 0))
        # rho = (max l - mean) / mean with the exact mean L/R, correctly rounded
        if Ltot > 0:
            mean = Fraction(Ltot, R)
            assert L.rho[b] == float((max(load) - mean) / mean)
        assert L.alpha[b] == float(Fraction(Ltot, E))


def test_spill_hand_example():
    """One hot rank with experts of load 5, 1, 3 (ids 0, 1, 2) and mean 4:
    ascending order 1, 3, 5 gives prefixes 1, 4, 9, cumulative excess 0, 0, 5,
    so only the heaviest expert spills, 5 tokens.  A second rank holds two
    experts of equal load 3 (ids 3, 4) against the same mean: the tie puts
    id 3 first, prefixes 3, 6 give spills 0 and 2."""
    R, E = 4, 7
    home = np.array([0, 0, 0, 1, 1, 2, 3], np.int32)
    # build n so that x = [5, 1, 3, 3, 3, 1, 0] -> loads [9, 6, 1, 0], L = 16, m = 4
    x = [5, 1, 3, 3, 3, 1, 0]
    ids = np.concatenate([np.full(c, e, np.int32) for e, c in enumerate(x)])
    ids = np.pad(ids, (0, 4 * 8 - ids.size), constant_values=-1).reshape(1, 4, 8)
    L = O.plan_loads(ids, home, E)
    np.testing.assert_array_equal(L.x[0], x)
    assert L.mean[0] == 4
    np.testing.assert_array_equal(L.excess[0], [5, 2, 0, 0])
    np.testing.assert_array_equal(L.spill[0], [5, 0, 0, 0, 2, 0, 0])


@pytest.mark.parametrize("seed", range(6))
def test_spill_invariants(seed):
    rng = np.random.default_rng(200 + seed)
    B, R, E, N = 2, int(rng.integers(2, 7)), int(rng.integers(3, 25)), 200
    # skewed ids so that some ranks are hot
    p = rng.dirichlet(np.full(E, 0.3))
    ids = rng.choice(E, size=(B, R, N), p=p).astype(np.int32)
    home = rng.integers(0, R, size=E).astype(np.int32)
    L = O.plan_loads(ids, home, E)
    for b in range(B):
        sp, x = L.spill[b], L.x[b]
        assert np.all(sp >= 0) and np.all(sp <= x)
        for r in range(R):
            mine = np.flatnonzero(home == r)
            # the spill of a rank's experts adds up to its excess
            assert sp[mine].sum() == L.excess[b, r]
            if mine.size:
                # experts are charged from the heaviest down: in ascending (load, id)
                # order the spill is zero on a prefix, then partial on at most one
                # expert, then the whole load
                order = sorted(mine, key=lambda e: (x[e], e))
                s = [int(sp[e]) for e in order]
                full = [int(sp[e]) == int(x[e]) for e in order]
                k = 0
                while k < len(s) and s[k] == 0:
                    k += 1
                if k < len(s) and not full[k]:
                    k += 1
                assert all(full[k:])


def test_spill_one_expert_per_rank_is_excess():
    """Identity home map (one expert per rank): spill_e = excess of its rank."""
    w = W.WORKLOADS[2]
    ids = W.problem_ids_host(w, 3)[None]
    L = O.plan_loads(ids, W.home_map(w), w.E)
    np.testing.assert_array_equal(L.spill[0], L.excess[0])


def test_zero_tokens():
    ids = np.zeros((1, 4, 0), np.int32)
    L = O.plan_loads(ids, np.arange(4, dtype=np.int32), 4)
    assert L.rho[0] == 0.0 and L.mean[0] == 0
    assert not L.excess.any() and not L.spare.any() and not L.spill.any()


def test_invalid_home_rejected():
    with pytest.raises(ValueError):
        O.plan_loads(np.zeros((1, 2, 3), np.int32), np.array([0, 2], np.int32), 2)
