"""Compile the C oracle into ``oracle/libmonomoe_oracle.so`` with gcc.

Flags keep IEEE semantics: no fast-math, no FMA contraction, so the two fp32 steps of
the quantiser (amax/448 and v/s) are single correctly rounded fp32 operations.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libmonomoe_oracle.so")


def build(verbose=False):
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fno-fast-math", "-ffp-contract=off",
           "-Wall", "-Wextra", "-o", LIB, os.path.join(HERE, "monomoe_oracle.c"), "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
