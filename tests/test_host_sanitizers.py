"""The library's host code (rg_api.cpp: planner, launch settings, argument checks, attention
workspace sizes) built with AddressSanitizer and UndefinedBehaviorSanitizer on the host side
only, driven over ~65 000 shape and setting combinations by tests/asan/plan_harness.cpp (kernel
launchers stubbed; no device work).  Any out-of-bounds access, overflow or other undefined
behaviour aborts the harness."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_host_code_clean_under_asan_and_ubsan(tmp_path):
    from paper_2609_25624_amd import build as b
    if not os.path.exists(b.HIPCC):
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "plan_harness")
    cmd = [b.HIPCC, "-x", "hip", "-std=c++17", "-O1", "-g", *b.DEVICE,
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined",
           os.path.join(ROOT, "paper_2609_25624_amd", "csrc", "rg_api.cpp"),
           os.path.join(ROOT, "tests", "asan", "plan_harness.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0 and r.stdout.startswith("ok:"), (r.stdout[-2000:], r.stderr[-4000:])
