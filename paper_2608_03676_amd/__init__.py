"""MI355X-native TAOT per-step replica planner.

Thin Python binding of libtaot.so (include/taot.h).  Every step of the path
runs in the library's HIP kernels; this module only checks tensor
dtypes/devices, allocates outputs and workspace with torch on the GPU, and
passes raw pointers plus the current HIP stream.  There is no CPU fallback:
calls raise if the library is not built or a tensor is not on the GPU.

Steps (paper Sec. 3.2 / Appendix A): plan_loads (expert-load histogram and
marginals), sinkhorn_batched (Phase 1), round_schedule (Phases 2 and 3);
plan_step chains them.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtaot.so")

ST_BAD_ID, ST_BAD_INPUT, ST_ZERO_MASS, ST_UNFILLED, ST_STREAMED = 0x1, 0x2, 0x4, 0x8, 0x10
SK_NO_COLCAP, SK_FORCE_STREAM, SK_NO_REGISTER, SK_WAVES_1, SK_DENSE, SK_LINEAR = 0x1, 0x2, 0x4, 0x8, 0x10, 0x20
SCH_NO_TOPO, SCH_NO_FLOW, SCH_ROW_PRIORITY = 0x1, 0x2, 0x4  # Phase-2 ablations (round_schedule flags)
STATUS_NAMES = {0: "ok", 1: "invalid argument", 2: "unsupported shape", 3: "workspace", 4: "launch"}

_lib = None
_P, _I32, _I64, _F32, _F64, _SZ, _U32 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                                         ctypes.c_double, ctypes.c_size_t, ctypes.c_uint32)


class TaotError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn}: {lib().taot_status_string(code).decode()} (status {code})")
        self.code = code


def lib():
    """Load libtaot.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        L.taot_status_string.restype = ctypes.c_char_p
        L.taot_status_string.argtypes = [ctypes.c_int]
        L.taot_plan_loads_workspace_size.restype = _SZ
        L.taot_plan_loads_workspace_size.argtypes = [_I32, _I32, _I32]
        L.taot_plan_loads.restype = ctypes.c_int
        L.taot_plan_loads.argtypes = [_P, _I32, _I32, _I64, _I32] + [_P] * 17 + [_P, _SZ, _P]
        L.taot_sinkhorn_workspace_size.restype = _SZ
        L.taot_sinkhorn_workspace_size.argtypes = [_I32, _I32]
        L.taot_sinkhorn_batched.restype = ctypes.c_int
        L.taot_sinkhorn_batched.argtypes = [_P, _P, _I32, _I32, _P, _I64, _F32, _I32, _U32, _P, _P, _P, _P,
                                            _P, _SZ, _P]
        L.taot_round_schedule_workspace_size.restype = _SZ
        L.taot_round_schedule_workspace_size.argtypes = [_I32, _I32, _I32, _I32]
        L.taot_round_schedule.restype = ctypes.c_int
        L.taot_round_schedule.argtypes = [_P] * 9 + [_I32] * 4 + [_F64, _I64, _U32] + [_P] * 6 + [_P, _SZ, _P]
        L.taot_topology_pref.restype = ctypes.c_int
        L.taot_topology_pref.argtypes = [_P, _I32, _P, _P]
        _lib = L
    return _lib


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dev(t: torch.Tensor, name: str, dtype) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _check(fn: str, code: int):
    if code != 0:
        raise TaotError(fn, code)


def _workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


@dataclasses.dataclass
class Loads:
    n: torch.Tensor        # [B][R][E] int32
    load_e: torch.Tensor   # [B][E] int64
    load_r: torch.Tensor   # [B][R] int64
    excess: torch.Tensor   # [B][R] int64
    spare: torch.Tensor    # [B][R] int64
    spill: torch.Tensor    # [B][E] int64
    supply: torch.Tensor   # [B][R] float32
    demand: torch.Tensor   # [B][R] float32
    rho: torch.Tensor      # [B] float64
    alpha: torch.Tensor    # [B] float64
    bad_ids: torch.Tensor  # [B] int64
    status: torch.Tensor   # [B] int32 (uint32 bits)
    hot_idx: Optional[torch.Tensor] = None   # [B][R] int32: ranks with excess > 0, ascending, then -1
    cold_idx: Optional[torch.Tensor] = None  # [B][R] int32: ranks with spare > 0, ascending, then -1
    hot_cnt: Optional[torch.Tensor] = None   # [B] int32
    cold_cnt: Optional[torch.Tensor] = None  # [B] int32


def plan_loads(ids: torch.Tensor, home: torch.Tensor, E: int, out: Optional[Loads] = None,
               workspace: Optional[torch.Tensor] = None, stream=None) -> Loads:
    """Steps 1-2: histogram n_re and the load marginals (taot_plan_loads)."""
    _dev(ids, "ids", torch.int32)
    _dev(home, "home", torch.int32)
    B, R, N = ids.shape
    dev = ids.device
    if out is None:
        out = Loads(*(torch.empty(s, dtype=d, device=dev) for s, d in (
            ((B, R, E), torch.int32), ((B, E), torch.int64), ((B, R), torch.int64), ((B, R), torch.int64),
            ((B, R), torch.int64), ((B, E), torch.int64), ((B, R), torch.float32), ((B, R), torch.float32),
            ((B,), torch.float64), ((B,), torch.float64), ((B,), torch.int64), ((B,), torch.int32))))
    if out.hot_idx is None:
        out.hot_idx = torch.empty((B, R), dtype=torch.int32, device=dev)
        out.cold_idx = torch.empty((B, R), dtype=torch.int32, device=dev)
        out.hot_cnt = torch.empty((B,), dtype=torch.int32, device=dev)
        out.cold_cnt = torch.empty((B,), dtype=torch.int32, device=dev)
    need = lib().taot_plan_loads_workspace_size(B, R, E)
    ws = workspace if workspace is not None else _workspace(need, dev)
    _check("taot_plan_loads", lib().taot_plan_loads(
        ids.data_ptr(), B, R, N, E, home.data_ptr(), out.n.data_ptr(), out.load_e.data_ptr(),
        out.load_r.data_ptr(), out.excess.data_ptr(), out.spare.data_ptr(), out.spill.data_ptr(),
        out.supply.data_ptr(), out.demand.data_ptr(), out.rho.data_ptr(), out.alpha.data_ptr(),
        out.bad_ids.data_ptr(), _ptr(out.hot_idx), _ptr(out.cold_idx), _ptr(out.hot_cnt), _ptr(out.cold_cnt),
        out.status.data_ptr(), ws.data_ptr(), ws.numel(), _stream(stream)))
    return out


@dataclasses.dataclass
class Flow:
    T: torch.Tensor        # [B][R][R] float32
    f: torch.Tensor        # [B][R] float32
    g: torch.Tensor        # [B][R] float32
    status: torch.Tensor   # [B] int32


def sinkhorn_batched(a: torch.Tensor, b: torch.Tensor, C: torch.Tensor, eps: float, iters: int,
                     flags: int = 0, out: Optional[Flow] = None, workspace: Optional[torch.Tensor] = None,
                     stream=None) -> Flow:
    """Step 3: batched Phase-1 Sinkhorn (taot_sinkhorn_batched).  C is [R][R]
    (shared) or [B][R][R]."""
    _dev(a, "a", torch.float32)
    _dev(b, "b", torch.float32)
    _dev(C, "C", torch.float32)
    B, R = a.shape
    if tuple(b.shape) != (B, R) or tuple(C.shape[-2:]) != (R, R) or C.dim() not in (2, 3):
        raise ValueError("shape mismatch among a, b, C")
    stride = 0 if C.dim() == 2 else R * R
    if C.dim() == 3 and C.shape[0] != B:
        raise ValueError("per-problem C needs B matrices")
    dev = a.device
    if out is None:
        out = Flow(torch.empty((B, R, R), dtype=torch.float32, device=dev),
                   torch.empty((B, R), dtype=torch.float32, device=dev),
                   torch.empty((B, R), dtype=torch.float32, device=dev),
                   torch.empty((B,), dtype=torch.int32, device=dev))
    need = lib().taot_sinkhorn_workspace_size(B, R)
    ws = workspace if workspace is not None else _workspace(need, dev)
    _check("taot_sinkhorn_batched", lib().taot_sinkhorn_batched(
        a.data_ptr(), b.data_ptr(), B, R, C.data_ptr(), stride, float(eps), int(iters), int(flags),
        _ptr(out.T), _ptr(out.f), _ptr(out.g), _ptr(out.status), ws.data_ptr(), ws.numel(), _stream(stream)))
    return out


@dataclasses.dataclass
class Schedule:
    slot_expert: torch.Tensor  # [B][R*K] int32
    slot_amount: torch.Tensor  # [B][R*K] int64
    X: torch.Tensor            # [B][R][R*K] int32
    unfilled: torch.Tensor     # [B] int64
    rounds_used: torch.Tensor  # [B][2] int32
    status: torch.Tensor       # [B] int32


def round_schedule(n, spill, spare, excess, alpha, home, T, Bpref, Bauct, K: int,
                   price_step: float = 2.0 ** -6, t_max: int = 0, out: Optional[Schedule] = None,
                   workspace: Optional[torch.Tensor] = None, stream=None, flags: int = 0) -> Schedule:
    """Steps 4-5: Phase-2 matching and Phase-3 auction (taot_round_schedule).
    flags: SCH_NO_TOPO / SCH_NO_FLOW drop a Phase-2 score term, SCH_ROW_PRIORITY matches
    from the experts' side (ablations)."""
    _dev(n, "n", torch.int32)
    for name, t in (("spill", spill), ("spare", spare), ("excess", excess)):
        _dev(t, name, torch.int64)
    _dev(alpha, "alpha", torch.float64)
    _dev(home, "home", torch.int32)
    _dev(T, "T", torch.float32)
    _dev(Bpref, "Bpref", torch.float64)
    _dev(Bauct, "Bauct", torch.float64)
    B, R, E = n.shape
    S = R * K
    dev = n.device
    if out is None:
        out = Schedule(torch.empty((B, S), dtype=torch.int32, device=dev),
                       torch.empty((B, S), dtype=torch.int64, device=dev),
                       torch.empty((B, R, S), dtype=torch.int32, device=dev),
                       torch.empty((B,), dtype=torch.int64, device=dev),
                       torch.empty((B, 2), dtype=torch.int32, device=dev),
                       torch.empty((B,), dtype=torch.int32, device=dev))
    need = lib().taot_round_schedule_workspace_size(B, R, E, K)
    ws = workspace if workspace is not None else _workspace(need, dev)
    _check("taot_round_schedule", lib().taot_round_schedule(
        n.data_ptr(), spill.data_ptr(), spare.data_ptr(), excess.data_ptr(), alpha.data_ptr(),
        home.data_ptr(), T.data_ptr(), Bpref.data_ptr(), Bauct.data_ptr(), B, R, E, K, float(price_step),
        int(t_max), int(flags), _ptr(out.slot_expert), _ptr(out.slot_amount), _ptr(out.X), _ptr(out.unfilled),
        _ptr(out.rounds_used), _ptr(out.status), ws.data_ptr(), ws.numel(), _stream(stream)))
    return out


def topology_pref(C: np.ndarray):
    """Host helper (taot_topology_pref): (Bpref, Bauct) fp64 [R][R] from a cost matrix."""
    C = np.ascontiguousarray(C, dtype=np.float32)
    R = C.shape[0]
    Bp = np.empty((R, R), np.float64)
    Ba = np.empty((R, R), np.float64)
    _check("taot_topology_pref", lib().taot_topology_pref(C.ctypes.data, R, Bp.ctypes.data, Ba.ctypes.data))
    return Bp, Ba


def workspace_bytes(B: int, R: int, E: int, K: int) -> dict:
    L = lib()
    return dict(plan_loads=L.taot_plan_loads_workspace_size(B, R, E),
                sinkhorn=L.taot_sinkhorn_workspace_size(B, R),
                round_schedule=L.taot_round_schedule_workspace_size(B, R, E, K))


@dataclasses.dataclass
class Plan:
    loads: Loads
    flow: Flow
    schedule: Schedule


def plan_step(ids, home, C, E: int, eps: float, iters: int, K: int, Bpref=None, Bauct=None,
              price_step: float = 2.0 ** -6, t_max: int = 0, stream=None, flags: int = 0) -> Plan:
    """One full planner step over all B problems (three enqueued calls, no sync)."""
    if Bpref is None or Bauct is None:
        Bp, Ba = topology_pref(C.detach().cpu().numpy() if isinstance(C, torch.Tensor) else C)
        Bpref = torch.from_numpy(Bp).to(ids.device)
        Bauct = torch.from_numpy(Ba).to(ids.device)
    loads = plan_loads(ids, home, E, stream=stream)
    flow = sinkhorn_batched(loads.supply, loads.demand, C, eps, iters, stream=stream)
    sched = round_schedule(loads.n, loads.spill, loads.spare, loads.excess, loads.alpha, home, flow.T,
                           Bpref, Bauct, K, price_step, t_max, stream=stream, flags=flags)
    return Plan(loads, flow, sched)


@dataclasses.dataclass
class Quality:
    load_after: torch.Tensor  # [B][R] int64 rank loads once the planned tokens moved
    rho_after: torch.Tensor   # [B] float64 (R * max load - L) / L, 0 if L = 0
    intra: torch.Tensor       # [B] int64 replicas hosted in their expert's home node
    inter: torch.Tensor       # [B] int64 replicas hosted in another node
    weighted: torch.Tensor    # [B] float64 intra + w_inter * inter


def plan_quality(load_r: torch.Tensor, home: torch.Tensor, sched: Schedule, K: int,
                 ranks_per_node: int = 8, w_inter: float = 3.0) -> Quality:
    """Plan-quality metrics of one schedule per problem (Sec. 4.1): the
    imbalance left after the planned tokens move from each expert's home rank
    to the ranks hosting its replicas, and the replicas placed inside and
    across nodes (node = rank // ranks_per_node), weighted intra + w_inter *
    inter.  Evaluation of a plan, not a planner step: plain tensor ops on the
    schedule's device."""
    se = sched.slot_expert.long()
    B, S = se.shape
    R = load_r.shape[1]
    valid = se >= 0
    moved = sched.X.sum(dim=1, dtype=torch.int64) * valid           # [B][S]
    host = (torch.arange(S, device=se.device) // K).expand(B, S)      # [B][S]
    h = home.long()[se.clamp(min=0)]                                  # [B][S]
    la = load_r.to(torch.int64).clone()
    la.scatter_add_(1, h, -moved)
    la.scatter_add_(1, host, moved)
    L = load_r.to(torch.int64).sum(1)
    lmax = la.max(1).values
    rho = torch.where(L > 0, (R * lmax - L).double() / L.clamp(min=1).double(),
                      torch.zeros_like(L, dtype=torch.float64))
    same = (h // ranks_per_node) == (host // ranks_per_node)
    intra = (valid & same).sum(1)
    inter = (valid & ~same).sum(1)
    return Quality(la, rho, intra, inter, intra.double() + w_inter * inter.double())


def plan_report(plan: Plan, home: torch.Tensor, K: int, problems=None, ranks_per_node: int = 8,
                w_inter: float = 3.0) -> str:
    """Text report of a finished plan, one block per chosen problem (layer),
    in the four parts of the planner log described in Appendix B.3:
    [1] every rank's load, ranks above the integer mean starred, and each
        expert that spills, with its home rank, load and spill;
    [2] one line per filled guest slot (expert, its home rank, the hosting
        rank and slot, same node or not, tokens the slot receives), then the
        copy counts and their weighted cost;
    [3] every rank's load once the planned tokens have moved;
    [4] rho and the largest rank load before and after, the share of all
        tokens sent to a replica, and the copy counts and cost.
    Formats on the host what the plan already holds."""
    L, sched = plan.loads, plan.schedule
    q = plan_quality(L.load_r, home, sched, K, ranks_per_node, w_inter)
    load_r, load_e = L.load_r.cpu().numpy(), L.load_e.cpu().numpy()
    excess, spill = L.excess.cpu().numpy(), L.spill.cpu().numpy()
    rho0, la, rho1 = L.rho.cpu().numpy(), q.load_after.cpu().numpy(), q.rho_after.cpu().numpy()
    se, X = sched.slot_expert.cpu().numpy(), sched.X.cpu().numpy()
    hm = home.cpu().numpy()
    B, R = load_r.shape
    problems = range(B) if problems is None else problems
    out = []

    def ranks(vals, marks=None):
        cells = [f"{r:4d}:{int(v):>9d}{'*' if marks is not None and marks[r] else ' '}" for r, v in enumerate(vals)]
        return ["   " + " ".join(cells[i:i + 8]) for i in range(0, len(cells), 8)]

    for b in problems:
        tot = int(load_r[b].sum())
        mean = tot / R if R else 0.0
        out.append(f"== plan report, problem {b}: R = {R}, E = {hm.shape[0]}, K = {K}, "
                   f"L = {tot}, mean {mean:.1f} ==")
        out.append("[1] load before routing (* hot rank: load above the integer mean)")
        out += ranks(load_r[b], excess[b] > 0)
        hot = np.nonzero(spill[b] > 0)[0]
        out.append(f"    hot experts (spill > 0): {len(hot)}")
        for e in hot:
            out.append(f"      expert {e:5d} on rank {hm[e]:4d}: load {int(load_e[b, e])}, spill {int(spill[b, e])}")
        out.append("[2] cloning plan")
        moved_tot, ni, no = 0, 0, 0
        for s_ in np.nonzero(se[b] >= 0)[0]:
            e, host = int(se[b, s_]), int(s_) // K
            moved = int(X[b, :, s_].sum())
            moved_tot += moved
            intra = hm[e] // ranks_per_node == host // ranks_per_node
            ni, no = ni + intra, no + (not intra)
            out.append(f"      expert {e:5d} (rank {hm[e]:4d}) -> slot {s_ % K} of rank {host:4d}: "
                       f"{'intra' if intra else 'inter'}-node, {moved} tokens")
        out.append(f"    topology: {ni} intra-node, {no} inter-node copies; weighted cost "
                   f"{ni + w_inter * no:.1f} (intra + {w_inter:g} x inter)")
        out.append("[3] projected load after routing")
        out += ranks(la[b])
        pk0, pk1 = int(load_r[b].max()), int(la[b].max())
        out.append("[4] summary")
        out.append(f"    imbalance rho {rho0[b]:.4f} -> {rho1[b]:.4f}; peak load {pk0} -> {pk1} "
                   f"({100.0 * (pk0 - pk1) / pk0 if pk0 else 0.0:.1f} % lower); rerouted {moved_tot} of "
                   f"{tot} tokens ({100.0 * moved_tot / tot if tot else 0.0:.2f} %); "
                   f"copies {ni} intra / {no} inter, weighted cost {ni + w_inter * no:.1f}")
    return "\n".join(out) + "\n"
