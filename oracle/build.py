"""Builds the CPU oracle (test infrastructure only) into oracle/libzo_oracle.so.

Plain C11 with OpenMP, -O2, no fast-math, no floating-point contraction: every
fp32 operation of the random-number contract rounds once, as written.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libzo_oracle.so")


def build(verbose: bool = False) -> str:
    tmp = f"{LIB}.{os.getpid()}.tmp"  # concurrent builds (parallel test workers) each write their own
    cmd = [
        "gcc", "-std=c11", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
        "-fPIC", "-shared", "-Wall", "-Wextra", "-Wno-unused-parameter",
        os.path.join(HERE, "zo_oracle.c"), "-o", tmp, "-lm",
    ]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
