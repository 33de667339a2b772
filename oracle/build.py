"""Compile the CPU oracle (plain C, host only) into oracle/librg_oracle.so.

Flags matter for what the oracle means: no contraction of a*b+c into FMA by
the compiler (-ffp-contract=off), no fast-math, and no -mfma for the
definitional oracle, so every fmaf in rg_oracle.c and rg_attn_oracle.c is the
C library's correctly rounded fused multiply-add.  The same-order vectorised
oracle (rg_oracle_fast.c) is compiled on its own with -mavx2 -mfma for its
explicit vector fused multiply-add intrinsics (still -ffp-contract=off).
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "librg_oracle.so")
FLAGS = ["-O2", "-std=c99", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
         "-fno-unsafe-math-optimizations"]


SOURCES = ["rg_oracle.c", "rg_attn_oracle.c"]
FAST_SOURCES = ["rg_oracle_fast.c"]
FAST_FLAGS = ["-std=c11", "-mavx2", "-mfma"]


def build(verbose: bool = False) -> str:
    objs = []
    for f in SOURCES + FAST_SOURCES:
        obj = os.path.join(HERE, f + ".o")
        extra = FAST_FLAGS if f in FAST_SOURCES else []
        cmd = ["gcc", *[a for a in FLAGS if a != "-shared"], *extra, "-c", os.path.join(HERE, f), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        objs.append(obj)
    cmd = ["gcc", "-shared", "-fopenmp", *objs, "-o", LIB + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    for o in objs:
        os.remove(o)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
