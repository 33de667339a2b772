"""A plain C99 program that calls librg through include/rg.h alone (no Python, no torch).

The program allocates device buffers with the HIP runtime, runs rg_linear on
five shapes (M = 1 GEMV-sized, ragged N and K, small batches, a 70-row batch),
and compares every output with the integer dot product on the host; the inputs
are small integers, so the exact sum is the only correct result.  It exits 0
when every check passes.  It is built by the package build step, in-tree.
"""
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "paper_2609_25624_amd", "examples", "linear_capi")


def test_example_source_uses_only_the_public_header():
    src = open(EXE + ".c").read()
    includes = [l.split()[1] for l in src.splitlines() if l.startswith("#include")]
    assert '"../../include/rg.h"' in includes
    assert not any("csrc" in i or "rg_kernels" in i for i in includes), includes


@pytest.mark.gpu
def test_c_program_runs_and_checks_exact_results():
    assert os.path.exists(EXE), "build the package first (paper_2609_25624_amd/build.py)"
    print(f"running {EXE}", flush=True)
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=100)
    sys.stdout.write(r.stdout)
    sys.stderr.write(r.stderr)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout
    assert len(re.findall(r": 0 of \d+ outputs wrong", r.stdout)) == 5
