"""Builds libtaot.so (all HIP sources, gfx950) and the benchmark's peak-probe
library libtaot_probes.so in-tree with hipcc.

Every floating-point operation rounds on its own (-ffp-contract=off; the
Sinkhorn kernels request fused multiply-adds explicitly), and packed-FP32
instructions are disabled.  Sources compile in parallel to objects under
_build/ and are then linked; `build(incremental=True)` reuses objects newer
than their source and headers (the default rebuilds everything).
"""
import concurrent.futures
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = ["csrc/api.hip", "csrc/loads.hip", "csrc/sinkhorn.hip", "csrc/sk_reg_w4g4.hip", "csrc/sk_reg_w2g8.hip",
           "csrc/sk_reg_w2g2.hip", "csrc/sk_dense.hip", "csrc/schedule.hip"]
LIB = os.path.join(HERE, "libtaot.so")
PROBES_LIB = os.path.join(HERE, "libtaot_probes.so")
OBJ_DIR = os.path.join(HERE, "_build")
FLAGS = ["-O3", "--offload-arch=gfx950", "-std=c++17", "-fPIC", "-ffp-contract=off",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wall",
         "-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(HERE, "csrc")]


def _run(cmd):
    r = subprocess.run(cmd, cwd=HERE, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("libtaot build failed: " + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    return "\n".join(l for l in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in l)


def build(verbose: bool = False, incremental: bool = False):
    os.makedirs(OBJ_DIR, exist_ok=True)
    headers = [os.path.join(ROOT, "include", "taot.h")] + glob.glob(os.path.join(HERE, "csrc", "*.h"))
    newest_header = max(os.path.getmtime(h) for h in headers)
    jobs = []
    for src in SOURCES:
        obj = os.path.join(OBJ_DIR, os.path.basename(src) + ".o")
        srcp = os.path.join(HERE, src)
        stale = (not incremental or not os.path.exists(obj) or os.path.getmtime(obj) < os.path.getmtime(srcp)
                 or os.path.getmtime(obj) < newest_header)
        jobs.append((["hipcc", *FLAGS, "-c", srcp, "-o", obj], stale, obj))
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(jobs)) as pool:
        logs = list(pool.map(lambda j: _run(j[0]) if j[1] else "", jobs))
    tmp = LIB + ".tmp"
    logs.append(_run(["hipcc", "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + [j[2] for j in jobs]))
    os.replace(tmp, LIB)
    # the benchmark's peak probes: a library of their own
    tmp = PROBES_LIB + ".tmp"
    logs.append(_run(["hipcc", *FLAGS, "-shared", os.path.join(HERE, "csrc", "probes.hip"), "-o", tmp]))
    os.replace(tmp, PROBES_LIB)
    if verbose:
        print("built", LIB)
        noise = "\n".join(l for l in logs if l)
        if noise:
            print(noise)


if __name__ == "__main__":
    build(verbose=True, incremental="--incremental" in sys.argv)
