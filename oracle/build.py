"""Compile the CPU oracle (plain C, fp64) into oracle/liboracle.so.

Test infrastructure: built next to the product so the checker exists, never
linked into it.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "fasgd_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

# No contraction into FMA and no fast-math, so every operation in the
# oracle's source is one IEEE fp64 operation.
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
          "-fno-fast-math", "-Wall", "-Wextra", "-Werror"]


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = ["gcc", *CFLAGS, "-o", tmp, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
