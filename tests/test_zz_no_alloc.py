"""taot_plan_loads_noalloc (the allocation-free variant of taot_plan_loads,
whose workspace is a fixed device array of the library) called through the
C-ABI: two calls in a row, the second on a smaller batch, each equal to
taot_plan_loads on the same input, output by output; shapes beyond its
scratch are refused with nothing enqueued."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2608_03676_amd as taot
import workloads as W

pytestmark = pytest.mark.gpu

_P, _I32, _I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64


def _lib():
    L = taot.lib()
    L.taot_plan_loads_noalloc.restype = ctypes.c_int
    L.taot_plan_loads_noalloc.argtypes = [_P, _I32, _I32, _I64, _I32] + [_P] * 17 + [_P]
    L.taot_plan_loads_noalloc_max_problems.restype = ctypes.c_size_t
    L.taot_plan_loads_noalloc_max_problems.argtypes = [_I32, _I32]
    return L


def _outputs(B, R, E, dev):
    return taot.Loads(*(torch.full(s, -7, dtype=d, device=dev) for s, d in (
        ((B, R, E), torch.int32), ((B, E), torch.int64), ((B, R), torch.int64), ((B, R), torch.int64),
        ((B, R), torch.int64), ((B, E), torch.int64), ((B, R), torch.float32), ((B, R), torch.float32),
        ((B,), torch.float64), ((B,), torch.float64), ((B,), torch.int64), ((B,), torch.int32),
        ((B, R), torch.int32), ((B, R), torch.int32), ((B,), torch.int32), ((B,), torch.int32))))


def _noalloc(ids, home, E, out):
    B, R, N = ids.shape
    stream = torch.cuda.current_stream().cuda_stream
    return _lib().taot_plan_loads_noalloc(
        ids.data_ptr(), B, R, N, E, home.data_ptr(), out.n.data_ptr(), out.load_e.data_ptr(),
        out.load_r.data_ptr(), out.excess.data_ptr(), out.spare.data_ptr(), out.spill.data_ptr(),
        out.supply.data_ptr(), out.demand.data_ptr(), out.rho.data_ptr(), out.alpha.data_ptr(),
        out.bad_ids.data_ptr(), out.hot_idx.data_ptr(), out.cold_idx.data_ptr(), out.hot_cnt.data_ptr(),
        out.cold_cnt.data_ptr(), out.status.data_ptr(), ctypes.c_void_p(stream))


def _same(a, b):
    for name in ("n", "load_e", "load_r", "excess", "spare", "spill", "supply", "demand", "rho", "alpha",
                 "bad_ids", "status", "hot_idx", "cold_idx", "hot_cnt", "cold_cnt"):
        x, y = getattr(a, name).cpu().numpy(), getattr(b, name).cpu().numpy()
        assert x.tobytes() == y.tobytes(), name


def test_noalloc_matches_plan_loads(gpu):
    # call 1: 12 problems of workload 1 (R = 64, E = 256), with skipped ids in
    # one row; call 2: 3 problems of workload 0 (R = 16, E = 64)
    for cfg, problems in ((1, list(range(12))), (0, [0, 0, 0])):
        w = W.WORKLOADS[cfg]
        print(f"[noalloc] workload {cfg}, {len(problems)} problems", flush=True)
        ids_np = np.stack([W.problem_ids_host(w, b) for b in problems])
        if cfg == 1:
            ids_np[3, 5, :7] = [-1, w.E, w.E + 5, -100, 2 ** 31 - 1, w.E, -2]
        ids = torch.from_numpy(ids_np).to(gpu)
        home = torch.from_numpy(W.home_map(w)).to(gpu)
        B, R, _ = ids.shape
        ref = taot.plan_loads(ids, home, w.E)
        out = _outputs(B, R, w.E, gpu)
        assert _noalloc(ids, home, w.E, out) == 0
        torch.cuda.synchronize()
        _same(out, ref)
        if cfg == 1:
            assert int(out.bad_ids[3]) == 7 and int(out.status[3]) == taot.ST_BAD_ID


def test_noalloc_refuses_beyond_scratch(gpu):
    L = _lib()
    R, E = 64, 256
    cap = L.taot_plan_loads_noalloc_max_problems(R, E)
    assert cap > 10000
    w = W.WORKLOADS[0]
    home = torch.from_numpy(W.home_map(w)).to(gpu)
    cap16 = L.taot_plan_loads_noalloc_max_problems(16, w.E)
    # a batch one problem beyond the scratch (ids of 8 tokens per row, every
    # output sized for it, so the call would be valid were it not for the
    # scratch): refused before anything is enqueued
    B = cap16 + 1
    ids = torch.zeros((B, 16, 8), dtype=torch.int32, device=gpu)
    out = _outputs(B, 16, w.E, gpu)
    assert _noalloc(ids, home, w.E, out) == 5  # TAOT_ERR_SCRATCH
    torch.cuda.synchronize()
    assert L.taot_status_string(5).decode().startswith("needs more than the fixed scratch")
    assert int(out.n.min()) == -7 and int(out.n.max()) == -7 and int(out.status.min()) == -7
    # the largest accepted batch runs
    out = _outputs(cap16, 16, w.E, gpu)
    assert _noalloc(ids[:cap16], home, w.E, out) == 0
    torch.cuda.synchronize()
    assert int(out.load_r.sum()) == cap16 * 16 * 8 and int(out.status.max()) == 0
