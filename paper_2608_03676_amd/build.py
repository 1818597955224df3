"""Builds libtaot.so (all HIP sources, gfx950) in-tree with hipcc.

Every floating-point operation rounds on its own (-ffp-contract=off; the
Sinkhorn kernels request fused multiply-adds explicitly), and packed-FP32
instructions are disabled."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = ["csrc/api.hip", "csrc/loads.hip", "csrc/sinkhorn.hip", "csrc/schedule.hip"]
LIB = os.path.join(HERE, "libtaot.so")
FLAGS = ["-O3", "--offload-arch=gfx950", "-std=c++17", "-fPIC", "-shared", "-ffp-contract=off",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wall",
         "-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(HERE, "csrc")]


def build(verbose: bool = False):
    tmp = LIB + ".tmp"
    cmd = ["hipcc", *FLAGS, "-o", tmp, *SOURCES]
    r = subprocess.run(cmd, cwd=HERE, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("libtaot build failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
        noise = [l for l in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in l]
        if noise:
            print("\n".join(noise))


if __name__ == "__main__":
    build(verbose=True)
