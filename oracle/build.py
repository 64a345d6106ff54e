"""Compile the CPU oracles (plain C, OpenMP) into oracle/liboracle_attn.so.

Test infrastructure: only tests, the smoke check and the benchmark's CPU
baseline load the result.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRCS = [os.path.join(HERE, "oracle_attn.c"), os.path.join(HERE, "oracle_opd.c")]
LIB = os.path.join(HERE, "liboracle_attn.so")


def build(verbose: bool = False) -> str:
    # -O2 without fast-math: plain IEEE double loops, libm exp.
    cmd = ["gcc", "-std=c11", "-O2", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-o", LIB + ".tmp", *SRCS, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
