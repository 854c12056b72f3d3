"""Builds the CPU oracle (test infrastructure only) into oracle/libmicro_oracle.so.

Plain gcc, -O2, no contraction of a*b+c into fused multiply-adds, no fast-math,
single translation unit.  Nothing under the product package links to it.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libmicro_oracle.so")
SRC = os.path.join(HERE, "micro_oracle.c")

CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
          "-fno-fast-math", "-Wall", "-Wextra", "-Werror"]


def build_oracle(verbose=False):
    """Compiles the oracle every time it is called; returns the library path."""
    tmp = LIB + ".tmp"
    cmd = ["gcc", *CFLAGS, "-o", tmp, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build_oracle(verbose=True))
