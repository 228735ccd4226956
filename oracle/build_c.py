"""Compile the oracle's C twin of the Jacobi sweep loop (test infrastructure).

``python -m oracle.build_c`` writes oracle/libjacobi_sweeps.so with gcc
(-O2, no fast-math, OpenMP over the disjoint pairs of a round).
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "jacobi_sweeps.c")
LIB = os.path.join(HERE, "libjacobi_sweeps.so")


def build(verbose=False):
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", SRC, "-o", LIB + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
