"""Build the C oracle (TEST INFRASTRUCTURE ONLY) into oracle/libkmq_oracle.so with gcc.

-ffp-contract=off keeps every fp32 expression exactly as written (no fused
multiply-adds other than the explicit fmaf calls).
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "kmq_oracle.c")
OUT = os.path.join(HERE, "libkmq_oracle.so")


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
           "-Wall", "-o", OUT + ".tmp", SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(OUT + ".tmp", OUT)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
