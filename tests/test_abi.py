"""CPU checks of the C-ABI library: it loads, exports every symbol the header
declares, rejects bad arguments on the host before touching the GPU, and its
host helper matches the oracle bit for bit.  No kernel runs here."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle as O
import paper_2608_03676_amd as taot
import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "taot.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(taot_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    names = _declared()
    assert {"taot_plan_loads", "taot_sinkhorn_batched", "taot_round_schedule", "taot_topology_pref",
            "taot_status_string"} <= set(names)
    lib = ctypes.CDLL(taot.LIB_PATH)
    for name in names:
        assert hasattr(lib, name), name


def test_probe_library_exports_its_header():
    """The benchmark's peak-probe library exports every symbol its header
    declares (no kernel runs here)."""
    src = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "taot_probes.h")).read(), flags=re.S)
    names = sorted(set(re.findall(r"\b(taot_probe_[a-z_]+)\s*\(", src)))
    assert names == ["taot_probe_exp", "taot_probe_fma", "taot_probe_hbm_read", "taot_probe_lds"]
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2608_03676_amd", "libtaot_probes.so"))
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings():
    L = taot.lib()
    for code in range(5):
        assert L.taot_status_string(code)
    assert b"unknown" in L.taot_status_string(99)


def test_workspace_sizes_monotone():
    L = taot.lib()
    assert L.taot_plan_loads_workspace_size(2, 16, 64) > 0
    assert L.taot_sinkhorn_workspace_size(4, 256) > L.taot_sinkhorn_workspace_size(2, 256)
    assert L.taot_round_schedule_workspace_size(8, 64, 256, 2) >= L.taot_round_schedule_workspace_size(8, 64, 256, 1)
    assert L.taot_sinkhorn_workspace_size(-1, 8) == 0


def _fake(n=1):
    return ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first


def test_host_validation_plan_loads():
    L = taot.lib()
    P = _fake()
    args = lambda B, R, N, E, ids=P, ws=P, wsb=1 << 30: L.taot_plan_loads(
        ids, B, R, N, E, P, P, P, P, P, P, P, None, None, None, P, None, None, None, None, None, None, ws, wsb,
        None)
    assert args(1, 0, 8, 4) == 1            # R <= 0
    assert args(1, 4, -1, 4) == 1           # N < 0
    assert args(1, 4, 8, 0) == 1            # E <= 0
    assert args(1, 2049, 8, 4) == 2         # R beyond TAOT_MAX_RANKS
    assert args(1, 4, 8, 40000) == 2        # E beyond TAOT_MAX_EXPERTS
    assert args(1, 4, 1 << 31, 4) == 2      # N beyond what an int32 count holds
    assert args(1, 4, 8, 4, ids=None) == 1  # null ids
    assert args(1, 4, 8, 4, ws=None) == 3   # no workspace
    assert args(1, 4, 8, 4, wsb=8) == 3     # workspace too small
    assert args(0, 4, 8, 4) == 0            # empty batch: nothing to do


def test_host_validation_sinkhorn():
    L = taot.lib()
    P = _fake()
    call = lambda B=1, R=4, stride=0, eps=0.1, iters=5, flags=0, ws=P, wsb=1 << 30: L.taot_sinkhorn_batched(
        P, P, B, R, P, stride, eps, iters, flags, P, None, None, None, ws, wsb, None)
    assert call(eps=0.0) == 1
    assert call(eps=float("nan")) == 1
    assert call(iters=0) == 1
    assert call(stride=7) == 1
    assert call(flags=0x80) == 1
    assert call(R=2049) == 2
    assert call(ws=None) == 3
    assert call(wsb=4) == 3
    assert call(B=0) == 0


def test_host_validation_round_schedule():
    L = taot.lib()
    P = _fake()
    call = lambda B=1, R=4, E=4, K=2, step=1.0 / 64, flags=0, ws=P, wsb=1 << 40: L.taot_round_schedule(
        P, P, P, P, P, P, P, P, P, B, R, E, K, step, 0, flags, P, P, P, P, None, None, ws, wsb, None)
    assert call(K=-1) == 1
    assert call(step=float("inf")) == 1
    assert call(flags=0x8) == 1          # unknown flag
    assert call(K=65) == 2
    assert call(ws=None) == 3
    assert call(wsb=16) == 3
    assert call(B=0) == 0


@pytest.mark.parametrize("cost", [("two_tier", 1.0, 4.0), ("three_tier", 1.0, 3.0, 8.0, 32),
                                  ("fat_tree", 1.0, 4.0, 16.0, 64)])
def test_topology_pref_matches_oracle_bitwise(cost):
    for R in (1, 2, 16, 128):
        C = W.cost_matrix_for(R, cost)
        Bp, Ba = taot.topology_pref(C)
        Op, Oa = O.topology_pref(C)
        assert Bp.tobytes() == Op.tobytes() and Ba.tobytes() == Oa.tobytes()
    rng = np.random.default_rng(3)
    C = rng.uniform(0.1, 9.0, (37, 37)).astype(np.float32)
    assert taot.topology_pref(C)[0].tobytes() == O.topology_pref(C)[0].tobytes()


def test_topology_pref_rejects_bad_costs():
    C = W.cost_matrix_for(4, ("two_tier", 1.0, 4.0))
    C[1, 2] = 0.0
    with pytest.raises(taot.TaotError):
        taot.topology_pref(C)


def test_noalloc_limits_on_host():
    """The allocation-free plan_loads refuses on the host, before any HIP
    call: invalid arguments, and batches whose workspace exceeds its fixed
    scratch (TAOT_ERR_SCRATCH); the limit shrinks with R and E."""
    L = taot.lib()
    L.taot_plan_loads_noalloc.restype = ctypes.c_int
    L.taot_plan_loads_noalloc.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                          ctypes.c_int32] + [ctypes.c_void_p] * 18
    L.taot_plan_loads_noalloc_max_problems.restype = ctypes.c_size_t
    L.taot_plan_loads_noalloc_max_problems.argtypes = [ctypes.c_int32, ctypes.c_int32]
    cap16 = L.taot_plan_loads_noalloc_max_problems(16, 64)
    cap_big = L.taot_plan_loads_noalloc_max_problems(2048, 32768)
    assert cap16 > cap_big > 100000
    assert L.taot_plan_loads_noalloc_max_problems(0, 64) == 0
    assert L.taot_plan_loads_noalloc_max_problems(16, 32769) == 0
    # the workspace of cap16 problems fits 1 MiB, one more does not
    assert L.taot_plan_loads_workspace_size(cap16, 16, 64) <= 1 << 20 < L.taot_plan_loads_workspace_size(cap16 + 1, 16, 64)
    p = [_fake()] * 17
    assert L.taot_plan_loads_noalloc(_fake(), cap16 + 1, 16, 8, 64, *p, None) == 5
    assert L.taot_status_string(5).startswith(b"needs more than the fixed scratch")
    assert L.taot_plan_loads_noalloc(None, 1, 16, 8, 64, *p, None) == 1  # ids NULL with N > 0
    assert L.taot_plan_loads_noalloc(_fake(), 1, 4096, 8, 64, *p, None) == 2  # R beyond the limit
