"""Host-side checks of the benchmark script: the one-GPU contract and the
sweep definitions (no GPU needed)."""
import os
import subprocess
import sys

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_hot_rank_panels_are_valid_workloads():
    sys.path.insert(0, ROOT)
    import bench
    pts = [p for _, points in bench.HOT_RANK_PANELS for p in points]
    assert {ep for ep, _, _ in pts} == set(W.LLEP_EP)
    assert {f for _, f, _ in pts} == set(W.LLEP_FRAC)
    assert {K for _, _, K in pts} == set(W.LLEP_K)
    for ep, frac, K in pts:
        w = W.llep_workload(ep, frac, K)
        assert w.R == ep and w.K == K and w.N == 8192 * 8
