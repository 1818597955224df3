"""Plan-quality metrics of the binding (tensor ops, here on the CPU) against
the oracle's plain loops: post-plan loads, rho after, intra / inter replica
counts and the weighted cost, on random schedules with empty slots and a
problem without load."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2608_03676_amd as taot


@pytest.mark.parametrize("seed,R,E,K,rpn", [(0, 16, 40, 2, 4), (1, 8, 8, 1, 8), (2, 64, 256, 4, 8), (3, 5, 3, 3, 2)])
def test_plan_quality_matches_oracle(seed, R, E, K, rpn):
    rng = np.random.default_rng(seed)
    B, S = 4, R * K
    load = rng.integers(0, 1000, size=(B, R)).astype(np.int64)
    load[1] = 0  # no load: rho after is 0
    home = rng.integers(0, R, size=E).astype(np.int32)
    se = rng.integers(-1, E, size=(B, S)).astype(np.int32)
    X = rng.integers(0, 5, size=(B, R, S)).astype(np.int32)
    X[se[:, None, :].repeat(R, 1) < 0] = 0  # empty slots receive nothing
    m = O.metrics(load, home, se, X, K, ranks_per_node=rpn, w_inter=3.0)
    sch = taot.Schedule(torch.from_numpy(se), torch.zeros((B, S), dtype=torch.int64), torch.from_numpy(X),
                        torch.zeros(B, dtype=torch.int64), torch.zeros((B, 2), dtype=torch.int32),
                        torch.zeros(B, dtype=torch.int32))
    q = taot.plan_quality(torch.from_numpy(load), torch.from_numpy(home), sch, K, ranks_per_node=rpn, w_inter=3.0)
    assert np.array_equal(q.load_after.numpy(), m["load_after"])
    assert q.rho_after.numpy().tobytes() == m["rho_after"].tobytes()
    assert np.array_equal(q.intra.numpy(), m["intra"]) and np.array_equal(q.inter.numpy(), m["inter"])
    assert q.weighted.numpy().tobytes() == m["weighted"].tobytes()
