"""Builds the oracle's shared library (plain C, gcc -O2, no hand SIMD).

Test infrastructure only: the product path never loads what this builds.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")
# -ffp-contract=off: every binary32 product is rounded on its own (no fused multiply-add)
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra", "-pthread", "-ffp-contract=off"]


def build(verbose: bool = False) -> str:
    cmd = ["gcc", *CFLAGS, SRC, "-o", LIB, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
