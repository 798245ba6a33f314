"""Build step for the CPU oracle shared library (test infrastructure only).

Compiles ``clq_oracle.c`` with gcc into ``libclq_oracle.so`` next to it:
``-O2 -fopenmp -ffp-contract=off`` with no fast-math and no intrinsics, so
every fp32 operation is a single IEEE-rounded add, subtract, multiply or
divide as written in the source.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "clq_oracle.c")
LIB = os.path.join(HERE, "libclq_oracle.so")

CFLAGS = ["-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
          "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra"]


def build(force=True):
    """Compile the oracle library; returns its path."""
    if not force and os.path.exists(LIB) and os.path.getmtime(LIB) >= os.path.getmtime(SRC):
        return LIB
    tmp = LIB + ".tmp"
    cmd = ["gcc", *CFLAGS, SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(force="--if-stale" not in sys.argv))
