"""Compile the CPU oracle (plain C, host only) into oracle/librg_oracle.so.

Flags matter for what the oracle means: no contraction of a*b+c into FMA by
the compiler (-ffp-contract=off), no fast-math, and no -mfma, so every fmaf
in the source is the C library's correctly rounded fused multiply-add.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "librg_oracle.so")
FLAGS = ["-O2", "-std=c99", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
         "-fno-unsafe-math-optimizations"]


SOURCES = ["rg_oracle.c", "rg_attn_oracle.c"]


def build(verbose: bool = False) -> str:
    srcs = [os.path.join(HERE, f) for f in SOURCES]
    cmd = ["gcc", *FLAGS, *srcs, "-o", LIB + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
