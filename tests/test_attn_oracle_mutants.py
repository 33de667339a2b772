"""Plant plausible mistakes in copies of the attention oracle and check its pins catch each one.

Each mutant is rg_attn_oracle.c with one edit, compiled alone into a temporary
library with the oracle's flags; it passes only if at least one check in
tests/attn_pins.py fails on it.  Nothing here touches a GPU.
"""
import ctypes
import os
import subprocess
import tempfile

import pytest

import oracle.build as ob
from tests import attn_pins as pins

SRC = os.path.join(os.path.dirname(ob.__file__), "rg_attn_oracle.c")

MUTANTS = {
    "position_segment_128": [("#define ATT_CHUNK 256", "#define ATT_CHUNK 128")],
    "sum_one_chain": [("        S = (j == 0) ? s : S + s;\n", "        S = (j == 0) ? s : S + s;\n        (void)0;\n"),
                      ("        float s = +0.0f;\n        for (int64_t l = l0; l < l1; ++l) s = s + e[l];",
                       "        float s = (j == 0) ? 0.0f : S;\n        for (int64_t l = l0; l < l1; ++l) s = s + e[l];\n        S = 0.0f;")],
    "no_max_subtraction": [("e[l] = rg_exp1(e[l] - m);", "e[l] = rg_exp1(e[l] - 0.0f * m);")],
    "exp_degree_6": [("float p = c[7];\n    for (int i = 6;", "float p = c[6];\n    for (int i = 5;")],
    "exp_truncates_k": [("const float k = rintf(u * L2E);", "const float k = truncf(u * L2E);")],
    "exp_single_ln2": [("    r = fmaf(-k, LN2_LO, r);\n", "")],
    "exp_cutoff_at_80": [("if (u < -87.0f) return 0.0f;", "if (u < -80.0f) return 0.0f;")],
    "divide_by_reciprocal": [("out[d] = N / S;", "out[d] = N * (1.0f / S);")],
    "scale_inside_dot": [("p = fmaf(q[d], attn_up(k[l * D + d]), p);", "p = fmaf(q[d] * scale, attn_up(k[l * D + d]), p);"),
                         ("e[l] = z * scale;", "e[l] = z;")],
    "gqa_mapping_modulo": [("const int64_t b = i / H, h = i % H, g = h / group;",
                            "const int64_t b = i / H, h = i % H, g = h % Hkv;")],
    "ignores_lengths": [("int64_t L = lens[b];", "int64_t L = Lmax; (void)lens;")],
    "value_chain_starts_at_minus_zero": [("float n = +0.0f;", "float n = -0.0f;")],
    "numerator_mul_add": [("n = fmaf(e[l], attn_up(v[l * D + d]), n);", "n = e[l] * attn_up(v[l * D + d]) + n;")],
}


def _build(name, edits, tmpdir):
    src = open(SRC).read()
    src2 = src
    for old, new in edits:
        assert old in src2, f"mutant {name}: edit anchor not found"
        src2 = src2.replace(old, new, 1)
    assert src2 != src
    c = os.path.join(tmpdir, f"attn_{name}.c")
    so = os.path.join(tmpdir, f"attn_{name}.so")
    open(c, "w").write(src2)
    subprocess.run(["gcc", *ob.FLAGS, c, "-o", so, "-lm"], check=True)
    return ctypes.CDLL(so)


@pytest.fixture(scope="module")
def tmpdir():
    with tempfile.TemporaryDirectory() as d:
        yield d


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_attention_pins_catch_mutant(name, tmpdir):
    L = _build(name, MUTANTS[name], tmpdir)
    caught = {}
    for check_name, check in pins.ALL_CHECKS.items():
        try:
            fails = check(L)
        except Exception as e:   # a crash in a check counts as caught
            fails = [repr(e)]
        if fails:
            caught[check_name] = fails[0]
            break
    assert caught, f"mutant {name} passed every pin"
