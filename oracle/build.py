"""Compile the CPU oracle (test infrastructure) into oracle/liboracle.so.

Plain gcc, no -ffast-math, no FP contraction, FTZ/DAZ untouched.  The target
is x86-64-v3 (AVX2) so the same shared object runs on any current server host.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

CFLAGS = [
    "-O3",
    "-std=c11",
    "-fPIC",
    "-shared",
    "-fopenmp",
    "-fno-fast-math",
    "-ffp-contract=off",
    "-march=x86-64-v3",
    "-Wall",
    "-Wextra",
]


def build(verbose: bool = False) -> str:
    cmd = ["gcc", *CFLAGS, SRC, "-o", LIB + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
