"""Build librg.so (HIP kernels + C-ABI) for gfx950 with hipcc, in-tree.

Floating-point flags are part of the method: -ffp-contract=off (no compiler
fusion of a*b+c), no fast-math, binary32 denormals kept, and packed FP32
instructions disabled, so each kernel performs exactly the operations its
source spells out.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "librg.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON = ["-O3", "-std=c++17", "-fPIC", "-ffp-contract=off", "-fno-fast-math",
          "-fno-gpu-flush-denormals-to-zero", "-Wall", "-Wno-unused-result"]
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
SOURCES = ["rg_kernels.hip", "rg_wtile.hip", "rg_attn.hip", "rg_api.cpp"]
# Negative controls (kernels that break the design rules on purpose, for the tests): a library of their own.
NEGCTL_LIB = os.path.join(HERE, "librg_negctl.so")
NEGCTL_SOURCES = ["rg_negctl.hip"]


# The comparison point (cast, then the vendor FP32 GEMM): a library of its own, so that
# librg.so has no BLAS dependency.  It calls librg's cast and rocBLAS.
BASELINE_LIB = os.path.join(HERE, "librg_baseline.so")
BASELINE_SOURCES = ["rg_baseline.cpp"]

# The read-bandwidth probe the benchmark's floors are measured with (not the product path).
PROBE_LIB = os.path.join(HERE, "librg_probe.so")
PROBE_SOURCES = ["rg_probe.hip"]

# A C program that uses the library through include/rg.h only (no Python).
EXAMPLE_SRC = os.path.join(HERE, "examples", "linear_capi.c")
EXAMPLE_BIN = os.path.join(HERE, "examples", "linear_capi")


def build(verbose: bool = False) -> str:
    _build_lib(SOURCES, LIB, verbose)
    _build_lib(NEGCTL_SOURCES, NEGCTL_LIB, verbose)
    _build_lib(PROBE_SOURCES, PROBE_LIB, verbose)
    rocm = os.path.dirname(os.path.dirname(os.path.realpath(HIPCC)))
    _build_lib(BASELINE_SOURCES, BASELINE_LIB, verbose,
               link=["-L" + HERE, "-lrg", "-L" + os.path.join(rocm, "lib"), "-lrocblas", "-Wl,-rpath,$ORIGIN",
                     "-Wl,-rpath," + os.path.join(rocm, "lib")])
    _build_example(verbose)
    return LIB


def _build_example(verbose):
    # host-only C99, built by the system C compiler: the C-ABI needs no HIP compiler on the caller's side
    rocm = os.path.dirname(os.path.dirname(os.path.realpath(HIPCC)))
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I" + os.path.join(rocm, "include"),
           EXAMPLE_SRC, "-L" + HERE, "-lrg", "-L" + os.path.join(rocm, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/..", "-Wl,-rpath," + os.path.join(rocm, "lib"), "-o", EXAMPLE_BIN + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("example build failed:\n" + r.stderr)
    os.replace(EXAMPLE_BIN + ".tmp", EXAMPLE_BIN)


def _build_lib(sources, lib, verbose, link=()):
    objs = []
    for src in sources:
        path = os.path.join(CSRC, src)
        obj = os.path.join(CSRC, src + ".o")
        cmd = [HIPCC, "-x", "hip", *COMMON, *DEVICE, "-c", path, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{err}")
        if err.strip() and verbose:
            print(err)
        objs.append(obj)
    cmd = [HIPCC, *DEVICE, "-shared", "-fPIC", *objs, *link, "-o", lib + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stderr)
    os.replace(lib + ".tmp", lib)


if __name__ == "__main__":
    print(build(verbose=True))
