"""The seeded input generator: SplitMix64 against its published outputs, the
inverse-CDF table, distinct top-k choices, and the hot-rank law of the
paper's scalability study (Sec. 4.4)."""
import math

import numpy as np
import pytest

import workloads as W


def test_splitmix64_published_outputs():
    """First outputs of SplitMix64 from state 0 (Steele, Lea and Flood, 2014),
    in the Python definition and in the C host twin."""
    ref = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    assert [W.splitmix64_at(0, i) for i in range(3)] == ref
    assert [W._host().gen_splitmix64_at(0, i) for i in range(3)] == ref


def test_threshold_table():
    wt = np.array([3.0, 0.0, 1.0, 4.0])
    thr = W.threshold_table(wt)
    assert thr.dtype == np.uint64 and int(thr[-1]) == 1 << 32
    assert np.all(np.diff(thr.astype(np.int64)) >= 0)
    assert int(thr[0]) == int(thr[1]) == int(3 / 8 * 2 ** 32)   # zero weight: empty interval


def test_distinct_choices_per_token():
    w = W.WORKLOADS[0]
    ids = W.problem_ids_host(w, 0).reshape(w.R, w.tokens, w.k)
    assert all(len(set(tok)) == w.k for row in ids for tok in row)
    assert ids.min() >= 0 and ids.max() < w.E


@pytest.mark.parametrize("ep,frac", [(4, 0.3), (16, 0.7), (32, 0.9)])
def test_hot_rank_law(ep, frac):
    """The hot rank's share of the choices is frac + (1 - frac) / R within six
    binomial standard deviations, its experts are hit uniformly, and every
    other expert is hit at rate (1 - frac) / E."""
    w = W.llep_workload(ep, frac)
    assert w.draw_shape == (w.tokens * w.k, 1) and w.N == 8192 * 8
    home = W.home_map(w)
    b = 3
    h = W.hot_rank(w, b)
    ids = W.problem_ids_host(w, b)
    n = ids.size
    cnt = np.bincount(ids.ravel(), minlength=w.E)
    p_hot = frac + (1 - frac) / ep
    share = cnt[home == h].sum() / n
    assert abs(share - p_hot) <= 6 * math.sqrt(p_hot * (1 - p_hot) / n), (share, p_hot)
    for mask, p in ((home == h, frac / (w.E // ep) + (1 - frac) / w.E), (home != h, (1 - frac) / w.E)):
        # chi-square over the experts of each group, against their common rate
        exp = p * n
        chi2 = ((cnt[mask] - exp) ** 2 / exp).sum()
        dof = mask.sum()
        assert chi2 <= dof + 6 * math.sqrt(2 * dof), (chi2, dof)


def test_hot_rank_seeding():
    w = W.llep_workload(16, 0.5)
    hots = [W.hot_rank(w, b) for b in range(w.B)]
    assert len(set(hots)) > 4 and all(0 <= h < 16 for h in hots)
    assert hots == [W.hot_rank(w, b) for b in range(w.B)]
    assert W.llep_workload(16, 0.5, K=8).master_seed == w.master_seed   # K does not change the ids
    assert W.llep_workload(16, 0.7).master_seed != w.master_seed


def test_hot_rank_workload_shape_and_cost():
    w = W.llep_workload(32, 0.5)
    C = W.cost_matrix(w)
    assert (w.B, w.R, w.E, w.eps) == (48, 32, 128, 3.0)
    assert np.all(np.diag(C) == 0) and C[0, 7] == 1.0 and C[0, 8] == 3.0
    assert np.array_equal(W.home_map(w), np.arange(128) // 4)
    with pytest.raises(ValueError):
        W.llep_workload(3, 0.5)
    with pytest.raises(ValueError):
        W.llep_workload(16, 1.5)
    with pytest.raises(ValueError):
        W.hot_rank(W.WORKLOADS[1], 0)
