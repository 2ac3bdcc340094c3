"""Build the CPU oracle shared libraries (test infrastructure only):
liboracle.so (serial) and liboracle_omp.so (the same functions with
list-level OpenMP entry points, for the benchmark's all-core baseline).

Compiled with gcc at -O2 and -ffp-contract=off so that every fp32 operation
is a single IEEE round-to-nearest-even step, as the oracle's definitions
require.  No fast-math, no vector intrinsics.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "bytecomp_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")
# the same functions with list-level OpenMP entry points (CPU baseline only)
SRC_OMP = os.path.join(HERE, "bytecomp_oracle_omp.c")
LIB_OMP = os.path.join(HERE, "liboracle_omp.so")


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-Wall", "-Wextra", "-o", LIB, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
           "-fPIC", "-shared", "-Wall", "-Wextra", "-o", LIB_OMP, SRC_OMP, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
