"""Plant plausible mistakes in copies of the CPU oracle and check the pins catch each one.

Each mutant is the oracle's C source with one edit, compiled into a temporary
library with the oracle's own flags.  A mutant passes this test only if at
least one pin in tests/oracle_pins.py fails on it.  Nothing here touches a GPU.
"""
import ctypes
import os
import re
import subprocess
import tempfile

import pytest

import oracle.build as ob
from tests import oracle_pins as pins

SRC = os.path.join(os.path.dirname(ob.__file__), "rg_oracle.c")

TREE_FOLD = r"""
float rg_oracle_dot(const float* x, const uint16_t* w, int64_t K) {
    float part[4096];
    int64_t J = 0;
    for (int64_t k0 = 0; k0 < K; k0 += RG_ORACLE_CHUNK, ++J) {
        const int64_t k1 = (k0 + RG_ORACLE_CHUNK < K) ? k0 + RG_ORACLE_CHUNK : K;
        float p = +0.0f;
        for (int64_t k = k0; k < k1; ++k) p = fmaf(x[k], up_bf16(w[k]), p);
        part[J] = p;
    }
    for (int64_t s = 1; s < J; s *= 2)
        for (int64_t i = 0; i + s < J; i += 2 * s) part[i] = part[i] + part[i + s];
    return part[0];
}
"""

MUTANTS = {
    "segment_128": [("#define RG_ORACLE_CHUNK 256", "#define RG_ORACLE_CHUNK 128")],
    "segment_512": [("#define RG_ORACLE_CHUNK 256", "#define RG_ORACLE_CHUNK 512")],
    "accumulator_starts_at_minus_zero": [("float p = +0.0f;", "float p = -0.0f;")],
    "reverse_order_in_segment": [("for (int64_t k = k0; k < k1; ++k)", "for (int64_t k = k1 - 1; k >= k0; --k)")],
    "drops_last_term_of_segment": [("for (int64_t k = k0; k < k1; ++k)", "for (int64_t k = k0; k < k1 - 1; ++k)")],
    "fold_from_plus_zero": [("if (j == 0)\n            y = p;\n        else\n            y = y + p;", "y = y + p;")],
    "double_accumulator": [("float p = +0.0f;", "double p = +0.0;"),
                           ("p = fmaf(x[k], up_bf16(w[k]), p);", "p = fma((double)x[k], (double)up_bf16(w[k]), p);")],
    "separate_multiply_add": [("p = fmaf(x[k], up_bf16(w[k]), p);", "p = x[k] * up_bf16(w[k]) + p;")],
    "transposed_output": [("const int64_t m = i / N, n = i % N;\n        y[i]", "const int64_t n = i / M, m = i % M;\n        y[i]")],
    "weight_row_stride_wrong": [("y[i] = rg_oracle_dot(x + m * K, w + n * K, K);",
                                 "y[i] = rg_oracle_dot(x + m * K, w + n * (K - 1), K);")],
    "flush_subnormal_weights": [("    memcpy(&f, &u, sizeof f);\n    return f;",
                                 "    memcpy(&f, &u, sizeof f);\n    return (fabsf(f) < 1.17549435e-38f) ? 0.0f : f;")],
    "upcast_shift_off_by_one": [("(uint32_t)b << 16", "(uint32_t)b << 15")],
    "tree_fold": "TREE",
    "bias_dropped": [("y[i] = d + b[n];", "y[i] = d;")],
    "bias_subtracted": [("y[i] = d + b[n];", "y[i] = d - b[n];")],
    "bias_in_double": [("y[i] = d + b[n];", "y[i] = (float)((double)d + (double)b[n] * 1.0000001);")],
    "f32w_weight_truncated_to_bf16": [("p = fmaf(x[k], w[k], p);", "p = fmaf(x[k], up_bf16((uint16_t)(f32_bits_of(w[k]) >> 16)), p);"),
                                      ("/* One output with FP32 weights", "static uint32_t f32_bits_of(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }\n/* One output with FP32 weights")],
    "f32w_flush_subnormal_weights": [("p = fmaf(x[k], w[k], p);", "p = fmaf(x[k], (fabsf(w[k]) < 1.17549435e-38f) ? 0.0f : w[k], p);")],
    "f32w_segment_512": [("const int64_t k1 = (k0 + RG_ORACLE_CHUNK < K) ? k0 + RG_ORACLE_CHUNK : K;\n        float p = +0.0f;\n        for (int64_t k = k0; k < k1; ++k) p = fmaf(x[k], w[k], p);",
                          "const int64_t k1 = (k0 + 2 * RG_ORACLE_CHUNK < K) ? k0 + 2 * RG_ORACLE_CHUNK : K;\n        float p = +0.0f;\n        for (int64_t k = k0; k < k1; ++k) p = fmaf(x[k], w[k], p);\n        k0 += RG_ORACLE_CHUNK;")],
}


def _build_mutant(name, edits, tmpdir):
    src = open(SRC).read()
    if edits == "TREE":
        src2 = re.sub(r"float rg_oracle_dot\(const float\* x.*?\n}\n", TREE_FOLD.strip() + "\n", src, count=1,
                      flags=re.S)
    else:
        src2 = src
        for old, new in edits:
            assert old in src2, f"mutant {name}: edit anchor not found"
            src2 = src2.replace(old, new, 1)
    assert src2 != src
    c = os.path.join(tmpdir, f"{name}.c")
    so = os.path.join(tmpdir, f"{name}.so")
    open(c, "w").write(src2)
    subprocess.run(["gcc", *ob.FLAGS, c, "-o", so, "-lm"], check=True)
    return ctypes.CDLL(so)


@pytest.fixture(scope="module")
def tmpdir():
    with tempfile.TemporaryDirectory() as d:
        yield d


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmpdir):
    L = _build_mutant(name, MUTANTS[name], tmpdir)
    caught = {}
    for check_name, check in pins.ALL_CHECKS.items():
        try:
            fails = check(L)
        except Exception as e:  # a crash in a check counts as caught
            fails = [repr(e)]
        if fails:
            caught[check_name] = fails[0]
    assert caught, f"mutant {name} passed every pin"
