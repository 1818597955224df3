"""Builds liboracle.so with gcc: -O2, OpenMP over problems, no floating-point
contraction and no fast-math, so every operation rounds as written."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))


def build(verbose: bool = False):
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", "-ffp-contract=off",
           "-fno-fast-math", "-o", "liboracle.so", "taot_oracle.c", "-lm"]
    r = subprocess.run(cmd, cwd=HERE, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("oracle build failed:\n" + r.stdout + r.stderr)
    if verbose:
        print("built", os.path.join(HERE, "liboracle.so"))


if __name__ == "__main__":
    build(verbose=True)
