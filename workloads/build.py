"""Builds the two twins of the input generator: a host shared library (gcc)
and a device shared library (hipcc, gfx950)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
HIP_FLAGS = ["-O3", "--offload-arch=gfx950", "-fPIC", "-shared", "-std=c++17",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd):
    r = subprocess.run(cmd, cwd=HERE, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("build failed: " + " ".join(cmd) + "\n" + r.stdout + r.stderr)


def build(verbose: bool = False):
    _run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", "-o",
          "libtaot_gen_host.so", "gen_ids.c"])
    _run(["hipcc", *HIP_FLAGS, "-o", "libtaot_gen_dev.so", "gen_ids_dev.hip"])
    if verbose:
        print("built", os.path.join(HERE, "libtaot_gen_host.so"), os.path.join(HERE, "libtaot_gen_dev.so"))


if __name__ == "__main__":
    build(verbose=True)
