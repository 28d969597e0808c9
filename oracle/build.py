"""Compile the CPU oracle (test infrastructure) into oracle/libkvmem_oracle.so.

Plain gcc, no fast-math and no FMA contraction, so every fp64 operation rounds
as written in kvmem_oracle.c.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "kvmem_oracle.c")
LIB = os.path.join(HERE, "libkvmem_oracle.so")


def build_oracle(verbose: bool = False) -> str:
    cmd = [
        "gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
        "-Wall", "-Wextra", "-shared", "-fPIC", SRC, "-o", LIB + ".tmp", "-lm",
    ]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build_oracle(verbose=True))
