"""Build the CPU oracle shared library (test infrastructure only).

The oracle is plain C compiled with IEEE semantics: no fast-math, no FMA
contraction, so fp32 division/rounding and fp64 accumulation are exactly
what the C source says.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "laq_oracle.c")
LIB = os.path.join(HERE, "liblaq_oracle.so")


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-O2", "-std=c11", "-fno-fast-math", "-ffp-contract=off",
           "-fopenmp", "-fPIC", "-shared", "-o", LIB + ".tmp", SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
