"""Build the CPU oracle shared library (test infrastructure only).

    python oracle/build.py

Compiles ``apex4_oracle.c`` with gcc into ``oracle/liboracle_apex4.so``.
No fast-math and no FP contraction: every rounding in the oracle is the one
its source code spells out.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "apex4_oracle.c")
LIB = os.path.join(HERE, "liboracle_apex4.so")


def build(verbose: bool = False) -> str:
    cmd = [
        "gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
        "-fno-fast-math", "-ffp-contract=off", "-Wall", "-Wextra",
        SRC, "-o", LIB + ".tmp", "-lm",
    ]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
