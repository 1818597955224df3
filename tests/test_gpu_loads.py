"""GPU parity of taot_plan_loads (histogram, loads, marginals, spill) with the
oracle: bit-exact on every integer output, exact fp64 rho/alpha."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2608_03676_amd as taot
import workloads as W
from helpers import oracle_inputs, random_loads_instance

pytestmark = pytest.mark.gpu


def _gpu_loads(ids, home, E):
    dev = torch.device("cuda:0")
    out = taot.plan_loads(torch.from_numpy(np.ascontiguousarray(ids)).to(dev),
                          torch.from_numpy(np.ascontiguousarray(home, dtype=np.int32)).to(dev), E)
    torch.cuda.synchronize()
    return {k: getattr(out, k).cpu().numpy() for k in out.__dataclass_fields__}


def _compare(g, ref, label=""):
    assert np.array_equal(g["n"], ref.n), f"{label} histogram"
    assert np.array_equal(g["load_e"], ref.x), f"{label} expert loads"
    assert np.array_equal(g["load_r"], ref.load), f"{label} rank loads"
    assert np.array_equal(g["excess"], ref.excess), f"{label} excess"
    assert np.array_equal(g["spare"], ref.spare), f"{label} spare"
    assert np.array_equal(g["spill"], ref.spill), f"{label} spill"
    assert np.array_equal(g["supply"], ref.excess.astype(np.float32)), f"{label} supply"
    assert np.array_equal(g["demand"], ref.spare.astype(np.float32)), f"{label} demand"
    assert g["rho"].tobytes() == ref.rho.tobytes(), f"{label} rho"
    assert g["alpha"].tobytes() == ref.alpha.tobytes(), f"{label} alpha"
    assert np.array_equal(g["bad_ids"], ref.bad), f"{label} bad ids"
    assert np.array_equal(g["status"].view(np.uint32), ref.status), f"{label} status"
    # the hot and cold sets (Sec. A.1) as ascending lists padded with -1
    for p in range(ref.excess.shape[0]):
        for name, vals in (("hot", ref.excess[p]), ("cold", ref.spare[p])):
            want = np.flatnonzero(vals > 0)
            got = g[name + "_idx"][p]
            assert g[name + "_cnt"][p] == want.size, f"{label} {name} count"
            assert np.array_equal(got[:want.size], want) and np.all(got[want.size:] == -1), f"{label} {name} list"


@pytest.mark.parametrize("cfg,problems", [(0, [0]), (1, list(range(58))), (2, [0, 1, 2, 3, 191, 383]),
                                          (3, [0, 977, 1951]), (4, [0, 63])])
def test_workloads(cfg, problems, gpu):
    w = W.WORKLOADS[cfg]
    print(f"[plan_loads parity] workload {cfg} problems {problems}", flush=True)
    ids, ref = oracle_inputs(w, problems)
    _compare(_gpu_loads(ids, W.home_map(w), w.E), ref, f"cfg{cfg}")


@pytest.mark.parametrize("seed", range(12))
def test_random_shapes(seed, gpu):
    rng = np.random.default_rng(seed)
    ids, home, E = random_loads_instance(rng)
    _compare(_gpu_loads(ids, home, E), O.plan_loads(ids, home, E))


# N = 4096 * k + 4 * t: k full batches of the vector path (1, 2, 3, 5; the
# batches alternate between two register sets) and a vector tail of t.
@pytest.mark.parametrize("R,E,N", [(1, 1, 5), (1, 7, 0), (3, 1, 13), (17, 5, 1), (64, 4097, 1003),
                                   (300, 64, 66), (5, 1023, 4096), (2, 32768, 64), (2048, 3, 2),
                                   (3, 40, 8260), (2, 384, 12292), (1, 64, 20480), (4, 9, 4092)])
def test_edge_shapes_with_bad_ids(R, E, N, gpu):
    rng = np.random.default_rng(R * 31 + E)
    B = 2
    ids = rng.integers(0, E, size=(B, R, N), dtype=np.int64)
    bad = rng.random(ids.shape) < 0.03
    ids[bad] = rng.choice([-1, E, E + 9, -(2**31), 2**31 - 1], size=int(bad.sum()))
    ids = ids.astype(np.int32)
    home = rng.integers(0, R, size=E).astype(np.int32)
    _compare(_gpu_loads(ids, home, E), O.plan_loads(ids, home, E), f"R{R} E{E} N{N}")


# Rows shorter than 2 * 65535 ids keep their counts as 16-bit pairs between
# the histogram and the expert sums, a count above 65534 in a spare word of its
# 256-expert block.  One expert per row takes nearly the whole row here, at
# the block edges and in the ragged last block; N = 131070 and up take the
# 32-bit form (there two experts of one pair can both pass 65534).
@pytest.mark.parametrize("E", [4, 260, 384, 512])
@pytest.mark.parametrize("N", [65535, 65536, 131068, 131070, 131072])
def test_counts_past_16_bits(E, N, gpu):
    rng = np.random.default_rng(E * 7 + N)
    hot = sorted({0, 1, 2, 3, 127, 128, 255, 256, 257, E - 2, E - 1} & set(range(E)))
    R = len(hot) + 1
    ids = rng.integers(0, E, size=(1, R, N), dtype=np.int64)
    for r, e in enumerate(hot):
        take = rng.random(N) < 0.9995 if r % 2 else np.ones(N, bool)
        ids[0, r, take] = e
        if r == 1:
            ids[0, r, :3] = [-1, E, E + 5]  # skipped ids next to a large count
    if N >= 131070:  # the two experts of a pair both above 65534
        ids[0, R - 1, :65535] = E - 2
        ids[0, R - 1, 65535:131070] = E - 1
    ids = ids.astype(np.int32)
    home = rng.integers(0, R, size=E).astype(np.int32)
    ref = O.plan_loads(ids, home, E)
    assert ref.n.max() >= 65535
    _compare(_gpu_loads(ids, home, E), ref, f"E{E} N{N}")


def test_unaligned_rows_use_scalar_path(gpu):
    """N not a multiple of 4 puts row starts off 16-byte alignment."""
    rng = np.random.default_rng(5)
    ids = rng.integers(0, 40, size=(3, 6, 1001), dtype=np.int32)
    home = (np.arange(40) % 6).astype(np.int32)
    _compare(_gpu_loads(ids, home, 40), O.plan_loads(ids, home, 40))


def test_all_experts_on_one_rank(gpu):
    rng = np.random.default_rng(6)
    ids = rng.integers(0, 50, size=(2, 8, 500), dtype=np.int32)
    home = np.zeros(50, np.int32)
    _compare(_gpu_loads(ids, home, 50), O.plan_loads(ids, home, 50))


def test_bad_home_sets_status(gpu):
    ids = np.zeros((2, 4, 8), np.int32)
    home = np.array([0, 1, 4, 2], np.int32)  # 4 is out of range for R = 4
    g = _gpu_loads(ids, home, 4)
    assert np.all(g["status"].view(np.uint32) & taot.ST_BAD_INPUT)
    assert not g["load_r"].any() and not g["spill"].any()
    assert not g["hot_cnt"].any() and not g["cold_cnt"].any()
    assert np.all(g["hot_idx"] == -1) and np.all(g["cold_idx"] == -1)


def test_deterministic(gpu):
    w = W.WORKLOADS[1]
    ids, _ = oracle_inputs(w, [0, 1, 2])
    a = _gpu_loads(ids, W.home_map(w), w.E)
    b = _gpu_loads(ids, W.home_map(w), w.E)
    for k in a:
        assert a[k].tobytes() == b[k].tobytes(), k


def test_device_generator_matches_host_twin(gpu):
    """The device twin of the input generator reproduces the host ids bit for bit."""
    dev = torch.device("cuda:0")
    for w, problems in ((W.WORKLOADS[0], [0]), (W.WORKLOADS[3], [5, 1900]), (W.WORKLOADS[4], [1]),
                        (W.llep_workload(32, 0.7), [0, 47])):
        thr, seeds = W.tables(w, problems)
        B = len(problems)
        ids = torch.empty((B, w.R, w.N), dtype=torch.int32, device=dev)
        W.gen_ids_device(torch.from_numpy(thr.view(np.int64)).to(dev), torch.from_numpy(seeds.view(np.int64)).to(dev),
                         B, w.E, w.R, *w.draw_shape, ids)
        torch.cuda.synchronize()
        got = ids.cpu().numpy()
        for q, b in enumerate(problems):
            rows = [0, w.R // 2, w.R - 1]
            for r in rows:
                ref = W.gen_ids_host(thr[q], int(seeds[q]), w.R, *w.draw_shape, r, r + 1)[0]
                assert np.array_equal(got[q, r], ref), (w.name, b, r)
