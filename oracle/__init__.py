"""ctypes binding of the double-precision CPU oracle (liboracle.so).

TEST INFRASTRUCTURE ONLY: imported by the tests, by the package smoke check
and by the benchmark's CPU-baseline leg.  The planner library and its Python
binding never import this module, and this module imports nothing from them.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")

EPS0 = 1e-12
ST_BAD_ID, ST_BAD_INPUT, ST_ZERO_MASS, ST_UNFILLED = 1, 2, 4, 8

_lib = None
_P = ctypes.c_void_p
_I32, _I64, _F64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            raise RuntimeError(f"{LIB} is not built; run oracle/build.py or __graft_entry__.build()")
        L = ctypes.CDLL(LIB)
        L.oracle_plan_loads.argtypes = [_P, _I32, _I32, _I64, _I32, _P] + [_P] * 11
        L.oracle_sinkhorn.argtypes = [_P, _P, _I32, _I32, _P, _I64, _F64, _I32, _I32, _F64, _I32,
                                      _P, _P, _P, _P, _P]
        L.oracle_topology_pref.argtypes = [_P, _I32, _P, _P]
        L.oracle_column_cap.argtypes = [_P, _P, _I32, _I32]
        L.oracle_max_threads.argtypes = []
        L.oracle_phase2.argtypes = [_P] * 7 + [_I32] * 4 + [ctypes.c_uint32] + [_P] * 3
        L.oracle_phase3.argtypes = [_P] * 4 + [_I32] * 4 + [_F64, _I64] + [_P] * 4
        L.oracle_metrics.argtypes = [_P] * 4 + [_I32] * 5 + [_F64] + [_P] * 5
        for f in (L.oracle_plan_loads, L.oracle_sinkhorn, L.oracle_topology_pref, L.oracle_column_cap,
                  L.oracle_phase2,
                  L.oracle_phase3, L.oracle_metrics, L.oracle_max_threads):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _check(rc, name):
    if rc != 0:
        raise ValueError(f"{name}: invalid arguments")


@dataclasses.dataclass
class Loads:
    n: np.ndarray        # [B][R][E] int32
    x: np.ndarray        # [B][E] int64 expert loads
    load: np.ndarray     # [B][R] int64 rank loads
    excess: np.ndarray   # [B][R] int64
    spare: np.ndarray    # [B][R] int64
    spill: np.ndarray    # [B][E] int64
    mean: np.ndarray     # [B] int64, floor(L / R)
    rho: np.ndarray      # [B] float64
    alpha: np.ndarray    # [B] float64
    bad: np.ndarray      # [B] int64
    status: np.ndarray   # [B] uint32


def plan_loads(ids, home, E: int) -> Loads:
    ids = _c(ids, np.int32)
    B, R, N = ids.shape
    home = _c(home, np.int32)
    out = Loads(np.empty((B, R, E), np.int32), np.empty((B, E), np.int64), np.empty((B, R), np.int64),
                np.empty((B, R), np.int64), np.empty((B, R), np.int64), np.empty((B, E), np.int64),
                np.empty(B, np.int64), np.empty(B, np.float64), np.empty(B, np.float64),
                np.empty(B, np.int64), np.empty(B, np.uint32))
    rc = lib().oracle_plan_loads(ids.ctypes.data, B, R, N, E, home.ctypes.data, out.n.ctypes.data,
                                 out.x.ctypes.data, out.load.ctypes.data, out.excess.ctypes.data,
                                 out.spare.ctypes.data, out.spill.ctypes.data, out.mean.ctypes.data,
                                 out.rho.ctypes.data, out.alpha.ctypes.data, out.bad.ctypes.data,
                                 out.status.ctypes.data)
    _check(rc, "oracle_plan_loads")
    return out


@dataclasses.dataclass
class Plan:
    T: np.ndarray        # [B][R][R] float64
    f: np.ndarray        # [B][R]
    g: np.ndarray        # [B][R]
    used: np.ndarray     # [B] int32
    status: np.ndarray   # [B] uint32


def sinkhorn(a, b, C, eps: float, iters: int, domain: str = "log", tol: float = 0.0,
             colcap: bool = True) -> Plan:
    a = _c(a, np.float64)
    b = _c(b, np.float64)
    if a.ndim == 1:
        a, b = a[None], b[None]
    B, R = a.shape
    C = _c(C, np.float64)
    stride = 0 if C.ndim == 2 else R * R
    out = Plan(np.empty((B, R, R)), np.empty((B, R)), np.empty((B, R)), np.empty(B, np.int32),
               np.empty(B, np.uint32))
    rc = lib().oracle_sinkhorn(a.ctypes.data, b.ctypes.data, B, R, C.ctypes.data, stride, eps, iters,
                               0 if domain == "log" else 1, tol, int(colcap), out.T.ctypes.data,
                               out.f.ctypes.data, out.g.ctypes.data, out.used.ctypes.data,
                               out.status.ctypes.data)
    _check(rc, "oracle_sinkhorn")
    return out


def column_cap(T, b) -> np.ndarray:
    """The column-cap step alone (Sec. A.2) on a copy of the plans T [B][R][R]."""
    T = np.array(T, dtype=np.float64, copy=True)
    b = _c(b, np.float64)
    if T.ndim == 2:
        T, b = T[None], b[None]
    B, R = b.shape
    _check(lib().oracle_column_cap(T.ctypes.data, b.ctypes.data, B, R), "oracle_column_cap")
    return T


def max_threads() -> int:
    """OpenMP threads the oracle's loops over problems may use."""
    return int(lib().oracle_max_threads())


def topology_pref(C):
    C = _c(C, np.float32)
    R = C.shape[0]
    Bp, Ba = np.empty((R, R)), np.empty((R, R))
    _check(lib().oracle_topology_pref(C.ctypes.data, R, Bp.ctypes.data, Ba.ctypes.data),
           "oracle_topology_pref")
    return Bp, Ba


SCH_NO_TOPO, SCH_NO_FLOW, SCH_ROW_PRIORITY = 0x1, 0x2, 0x4  # Phase-2 ablations


def phase2(spill, spare, excess, alpha, home, T32, Bpref, K: int, flags: int = 0):
    spill = _c(spill, np.int64)
    if spill.ndim == 1:
        spill, spare, excess = spill[None], _c(spare, np.int64)[None], _c(excess, np.int64)[None]
        alpha = np.atleast_1d(alpha)
        T32 = _c(T32, np.float32)[None]
    spare, excess = _c(spare, np.int64), _c(excess, np.int64)
    alpha = _c(alpha, np.float64)
    T32 = _c(T32, np.float32)
    home = _c(home, np.int32)
    Bpref = _c(Bpref, np.float64)
    B, E = spill.shape
    R = spare.shape[1]
    se = np.empty((B, R * K), np.int32)
    sa = np.empty((B, R * K), np.int64)
    used = np.empty(B, np.int32)
    rc = lib().oracle_phase2(spill.ctypes.data, spare.ctypes.data, excess.ctypes.data, alpha.ctypes.data,
                             home.ctypes.data, T32.ctypes.data, Bpref.ctypes.data, B, R, E, K, flags,
                             se.ctypes.data, sa.ctypes.data, used.ctypes.data)
    _check(rc, "oracle_phase2")
    return se, sa, used


def phase3(n, slot_expert, slot_amount, Bauct, K: int, eta: float = 2.0 ** -6, t_max: int = 0):
    n = _c(n, np.int32)
    if n.ndim == 2:
        n = n[None]
        slot_expert = _c(slot_expert, np.int32)[None]
        slot_amount = _c(slot_amount, np.int64)[None]
    slot_expert, slot_amount = _c(slot_expert, np.int32), _c(slot_amount, np.int64)
    Bauct = _c(Bauct, np.float64)
    B, R, E = n.shape
    X = np.empty((B, R, R * K), np.int32)
    unfilled = np.empty(B, np.int64)
    rounds = np.empty(B, np.int64)
    status = np.empty(B, np.uint32)
    rc = lib().oracle_phase3(n.ctypes.data, slot_expert.ctypes.data, slot_amount.ctypes.data,
                             Bauct.ctypes.data, B, R, E, K, eta, t_max, X.ctypes.data,
                             unfilled.ctypes.data, rounds.ctypes.data, status.ctypes.data)
    _check(rc, "oracle_phase3")
    return X, unfilled, rounds, status


def metrics(load, home, slot_expert, X, K: int, ranks_per_node: int = 8, w_inter: float = 3.0):
    load = _c(load, np.int64)
    slot_expert, X = _c(slot_expert, np.int32), _c(X, np.int32)
    home = _c(home, np.int32)
    B, R = load.shape
    E = home.shape[0]
    la = np.empty((B, R), np.int64)
    rho = np.empty(B)
    intra, inter = np.empty(B, np.int64), np.empty(B, np.int64)
    wt = np.empty(B)
    rc = lib().oracle_metrics(load.ctypes.data, home.ctypes.data, slot_expert.ctypes.data, X.ctypes.data,
                              B, R, E, K, ranks_per_node, w_inter, la.ctypes.data, rho.ctypes.data,
                              intra.ctypes.data, inter.ctypes.data, wt.ctypes.data)
    _check(rc, "oracle_metrics")
    return dict(load_after=la, rho_after=rho, intra=intra, inter=inter, weighted=wt)
