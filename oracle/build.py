"""Builds the CPU oracle shared library (test infrastructure only).

    python -m oracle.build

Plain g++ with OpenMP; no BLAS.  The flags are generic x86-64-v3 so that a
library built in one container also runs on another host.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "bp_oracle.cpp")
OUT = os.path.join(HERE, "liboracle.so")


def build(verbose: bool = False) -> str:
    cmd = ["g++", "-O3", "-march=x86-64-v3", "-fPIC", "-shared", "-fopenmp", "-std=c++17",
           "-Wall", "-Wextra", SRC, "-o", OUT + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(OUT + ".tmp", OUT)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
