"""Seeded synthetic workloads for the TAOT per-step planner.

This module only produces inputs: routing ids, the expert->rank home map, the
rank-to-rank cost matrix and the run parameters.  It holds none of the
planner's arithmetic and is the only code that both the oracle side and the
HIP side of the tests consume.

Five workloads are defined (indices 0-4).  Ranks exist only as data; rank r
sits on node r // 8.  Expert ids of each (problem, source rank) row are drawn
per token as k = 8 distinct experts by successive sampling without
replacement from a Zipf law over a seeded permutation of the experts (see
gen_ids.h for the exact counter-based definition).

A second family, `llep_workload(ep, frac, K)`, follows the imbalance
construction of the paper's scalability study (Sec. 4.4): in every problem a
seeded hot rank receives a fraction `frac` of the routing choices and the
rest go to uniformly random experts, on a Qwen3-30B-A3B-shaped layer (128
experts, top-8, 48 layers) at EP 4-32, with the paper's two-tier cost
(1 inside a node, lambda = 3 across nodes) and eps = lambda.

The paper's own routing came from Qwen3-30B-A3B on the Pile test split
(Sec. 4.1); neither is available here, so these synthetic loads stand in
for it.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_HOST = os.path.join(HERE, "libtaot_gen_host.so")
LIB_DEV = os.path.join(HERE, "libtaot_gen_dev.so")

SPLITMIX_GAMMA = 0x9E3779B97F4A7C15
MASK64 = (1 << 64) - 1


def splitmix64_at(seed: int, i: int) -> int:
    """i-th output of SplitMix64 started from state `seed` (same as gen_ids.h)."""
    z = (seed + (i + 1) * SPLITMIX_GAMMA) & MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


@dataclasses.dataclass(frozen=True)
class Workload:
    index: int
    name: str
    B: int                 # problems (MoE layers x micro-batches)
    R: int                 # EP ranks
    E: int                 # experts
    tokens: int            # tokens per source rank
    k: int                 # top-k
    home: str              # "block" (e // (E/R)), "identity" (e), "roundrobin" (e mod R)
    zipf: tuple            # ("fixed", s) | ("uniform", lo, hi) | ("hot_rank", frac)
    spike: Optional[tuple]  # (fraction of experts, factor) or None
    cost: tuple            # ("two_tier", intra, inter) | ("three_tier", node, rack, far, rack_ranks)
                           # | ("fat_tree", node, leaf, far, leaf_ranks)
    eps: float             # absolute entropic regulariser
    iters: int             # Sinkhorn iterations
    K: int = 2             # guest slots per rank
    price_step: float = 2.0 ** -6
    distinct: bool = True  # a token's k choices are distinct experts (else drawn independently)
    seed: Optional[int] = None  # master seed (default 20260801 + index)

    @property
    def N(self) -> int:
        """Routing ids per (problem, source rank) row."""
        return self.tokens * self.k

    @property
    def draw_shape(self):
        """(tokens, choices per token) as passed to the generator: independent
        choices are k draws of one choice each, so no choice is ever redrawn."""
        return (self.tokens, self.k) if self.distinct else (self.tokens * self.k, 1)

    @property
    def master_seed(self) -> int:
        return 20260801 + self.index if self.seed is None else self.seed


WORKLOADS = [
    Workload(0, "single layer, R=16 (2 nodes x 8), 64 experts, 4096 tokens top-8",
             B=1, R=16, E=64, tokens=256, k=8, home="block", zipf=("fixed", 1.0), spike=None,
             cost=("two_tier", 1.0, 4.0), eps=0.2, iters=200),
    Workload(1, "DeepSeek-V3-shaped: 58 layers, R=64, 256 experts",
             B=58, R=64, E=256, tokens=16384, k=8, home="block", zipf=("fixed", 1.2), spike=None,
             cost=("two_tier", 1.0, 4.0), eps=0.08, iters=500),
    Workload(2, "Qwen3-MoE-shaped: 48 layers x 8 micro-batches, R=128, 128 experts",
             B=384, R=128, E=128, tokens=8192, k=8, home="identity", zipf=("uniform", 0.8, 1.5),
             spike=None, cost=("three_tier", 1.0, 3.0, 8.0, 32), eps=0.08, iters=1000),
    Workload(3, "Kimi-K2-shaped: 61 layers x 32 micro-batches, R=256, 384 experts",
             B=1952, R=256, E=384, tokens=8192, k=8, home="roundrobin", zipf=("fixed", 1.3),
             spike=(0.1, 5.0), cost=("three_tier", 1.0, 3.0, 8.0, 32), eps=0.08, iters=1000),
    Workload(4, "stress: 64 problems, R=1024, 4096 experts, 2^26 ids per problem",
             B=64, R=1024, E=4096, tokens=8192, k=8, home="block", zipf=("fixed", 1.5), spike=None,
             cost=("fat_tree", 1.0, 4.0, 16.0, 64), eps=0.08, iters=2000),
]


LLEP_EP = (4, 8, 16, 32)
LLEP_FRAC = (0.3, 0.5, 0.7, 0.9)
LLEP_K = (1, 2, 4, 8, 16)


def llep_workload(ep: int, frac: float, K: int = 2) -> Workload:
    """Hot-rank workload of the paper's scalability study (Sec. 4.4) at EP
    degree `ep` and hot fraction `frac`: 48 problems (one per MoE layer of a
    Qwen3-30B-A3B-shaped model: 128 experts in blocks of 128 / ep per rank,
    top-8), 8192 tokens per rank (a 32768-token sequence over 4-way tensor
    parallelism, Appendix B), cost 1 inside a node of 8 ranks and lambda = 3
    across nodes (Sec. A.1), eps = lambda (Sec. A.2), 200 iterations."""
    if ep < 1 or 128 % ep or not 0.0 <= frac <= 1.0:
        raise ValueError(f"llep_workload: ep must divide 128 and 0 <= frac <= 1 (got {ep}, {frac})")
    return Workload(100 + ep, f"LLEP-style hot rank: EP{ep}, {round(100 * frac)}% to one rank, K={K}",
                    B=48, R=ep, E=128, tokens=8192, k=8, home="block", zipf=("hot_rank", float(frac)),
                    spike=None, cost=("two_tier", 1.0, 3.0), eps=3.0, iters=200, K=K, distinct=False,
                    seed=20260901 + 1000 * ep + round(1000 * frac))


def hot_rank(w: Workload, b: int) -> int:
    """The overloaded rank of problem b of a hot-rank workload."""
    if w.zipf[0] != "hot_rank":
        raise ValueError("hot_rank: not a hot-rank workload")
    rng = np.random.Generator(np.random.PCG64([w.master_seed, b]))
    return int(rng.integers(w.R))


def home_map(w: Workload) -> np.ndarray:
    e = np.arange(w.E, dtype=np.int64)
    if w.home == "block":
        h = e // (w.E // w.R)
    elif w.home == "identity":
        h = e
    elif w.home == "roundrobin":
        h = e % w.R
    else:
        raise ValueError(w.home)
    return h.astype(np.int32)


def cost_matrix(w: Workload) -> np.ndarray:
    return cost_matrix_for(w.R, w.cost)


def cost_matrix_for(R: int, cost: tuple) -> np.ndarray:
    """C[i][j] (fp32): 0 on the diagonal, topology tiers elsewhere; node = rank // 8."""
    r = np.arange(R)
    node = r // 8
    same_node = node[:, None] == node[None, :]
    kind = cost[0]
    if kind == "two_tier":
        C = np.where(same_node, cost[1], cost[2])
    elif kind in ("three_tier", "fat_tree"):
        group = r // cost[4]
        same_group = group[:, None] == group[None, :]
        C = np.where(same_node, cost[1], np.where(same_group, cost[2], cost[3]))
    else:
        raise ValueError(kind)
    C = C.astype(np.float32)
    np.fill_diagonal(C, 0.0)
    return C


def problem_seed(w: Workload, b: int) -> int:
    return splitmix64_at(w.master_seed, b)


def expert_weights(w: Workload, b: int) -> np.ndarray:
    """Unnormalised routing weight of each expert for problem b (fp64).

    Hot-rank law: a choice goes with probability frac to a uniformly chosen
    expert of the hot rank and otherwise to a uniformly chosen expert of all
    E, so the hot rank's expected share of the choices is
    frac + (1 - frac) / R when every rank homes E / R experts."""
    if w.zipf[0] == "hot_rank":
        frac = w.zipf[1]
        hot = home_map(w) == hot_rank(w, b)
        return np.full(w.E, (1.0 - frac) / w.E) + np.where(hot, frac / hot.sum(), 0.0)
    rng = np.random.Generator(np.random.PCG64([w.master_seed, b]))
    perm = rng.permutation(w.E)
    if w.zipf[0] == "fixed":
        s = w.zipf[1]
    else:
        s = rng.uniform(w.zipf[1], w.zipf[2])
    wt = np.empty(w.E, dtype=np.float64)
    wt[perm] = (np.arange(w.E, dtype=np.float64) + 1.0) ** (-s)
    if w.spike is not None:
        n_spike = int(round(w.spike[0] * w.E))
        spiked = rng.choice(w.E, size=n_spike, replace=False)
        wt[spiked] *= w.spike[1]
    return wt


def threshold_table(weights: np.ndarray) -> np.ndarray:
    """uint64 inverse-CDF table: expert = min{e : u < thr[e]} for u in [0, 2^32)."""
    p = np.asarray(weights, dtype=np.float64)
    cum = np.cumsum(p / p.sum())
    thr = np.floor(np.minimum(cum, 1.0) * 2.0 ** 32).astype(np.uint64)
    thr[-1] = np.uint64(1 << 32)
    return thr


def tables(w: Workload, problems=None):
    """(thr [P][E] uint64, seeds [P] uint64) for the given problem indices."""
    problems = range(w.B) if problems is None else problems
    thr = np.stack([threshold_table(expert_weights(w, b)) for b in problems])
    seeds = np.array([problem_seed(w, b) for b in problems], dtype=np.uint64)
    return np.ascontiguousarray(thr), seeds


_host_lib = None
_dev_lib = None


def _host():
    global _host_lib
    if _host_lib is None:
        if not os.path.exists(LIB_HOST):
            raise RuntimeError(f"{LIB_HOST} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_HOST)
        lib.gen_ids_host.restype = ctypes.c_int
        lib.gen_ids_host.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64, ctypes.c_int32,
                                     ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_void_p]
        lib.gen_splitmix64_at.restype = ctypes.c_uint64
        lib.gen_splitmix64_at.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        _host_lib = lib
    return _host_lib


def gen_ids_host(thr: np.ndarray, seed: int, R: int, T: int, k: int, r0: int = 0,
                 r1: Optional[int] = None) -> np.ndarray:
    """ids [r1-r0][T*k] int32 for one problem, on the host."""
    r1 = R if r1 is None else r1
    thr = np.ascontiguousarray(thr, dtype=np.uint64)
    out = np.empty(((r1 - r0), T * k), dtype=np.int32)
    rc = _host().gen_ids_host(thr.ctypes.data, thr.shape[0], ctypes.c_uint64(int(seed)), R, T, k, r0,
                              r1, out.ctypes.data)
    if rc != 0:
        raise ValueError("gen_ids_host: invalid arguments")
    return out


def problem_ids_host(w: Workload, b: int, r0: int = 0, r1: Optional[int] = None) -> np.ndarray:
    thr, seeds = tables(w, [b])
    return gen_ids_host(thr[0], int(seeds[0]), w.R, *w.draw_shape, r0, r1)


def _dev():
    global _dev_lib
    if _dev_lib is None:
        if not os.path.exists(LIB_DEV):
            raise RuntimeError(f"{LIB_DEV} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_DEV)
        lib.gen_ids_device.restype = ctypes.c_int
        lib.gen_ids_device.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                       ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                       ctypes.c_void_p]
        _dev_lib = lib
    return _dev_lib


def workload_ids_device(w: Workload, dev, problems=None):
    """ids [P][R][N] int32 on `dev` for the given problems (all by default),
    made by the device twin."""
    import torch
    thr, seeds = tables(w, problems)
    P = len(seeds)
    ids = torch.empty((P, w.R, w.N), dtype=torch.int32, device=dev)
    gen_ids_device(torch.from_numpy(thr.view(np.int64)).to(dev), torch.from_numpy(seeds.view(np.int64)).to(dev),
                   P, w.E, w.R, *w.draw_shape, ids)
    return ids


def gen_ids_device(thr_dev, seeds_dev, B: int, E: int, R: int, T: int, k: int, ids_dev, stream=None):
    """Fill ids_dev (torch int32 [B][R][T*k] on the GPU) with the device twin."""
    import torch
    assert thr_dev.dtype == torch.uint64 or thr_dev.dtype == torch.int64
    assert ids_dev.dtype == torch.int32 and ids_dev.is_contiguous()
    assert ids_dev.numel() == B * R * T * k and thr_dev.numel() == B * E and seeds_dev.numel() == B
    s = torch.cuda.current_stream().cuda_stream if stream is None else stream
    rc = _dev().gen_ids_device(thr_dev.data_ptr(), seeds_dev.data_ptr(), B, E, R, T, k,
                               ids_dev.data_ptr(), ctypes.c_void_p(s))
    if rc != 0:
        raise RuntimeError("gen_ids_device failed")

