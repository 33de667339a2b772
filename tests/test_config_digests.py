"""The stored full-output digests of the batched and large workloads (tests/golden/config_digests.json,
written by tests/golden/make_config_digests.py from the oracle alone) are re-derived here on the CPU,
so the oracle and the input generator have not drifted from them.  The GPU tests hash rg_linear's
full outputs against the same digests."""
import json
import os

import pytest

import oracle
from tests.golden import make_config_digests as mk

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "config_digests.json")


def test_stored_cases_are_the_generator_cases():
    stored = json.load(open(GOLDEN))["cases"]
    assert sorted(stored) == sorted(c["name"] for c in mk.CASES)
    for c in mk.CASES:
        assert {k: stored[c["name"]][k] for k in ("M", "N", "K", "std", "layer", "xrows")} == \
               {k: c[k] for k in ("M", "N", "K", "std", "layer", "xrows")}


@pytest.mark.slow
@pytest.mark.skipif(not oracle.fast_supported(), reason="host CPU lacks AVX2/FMA")
def test_oracle_reproduces_every_stored_config_digest():
    stored = json.load(open(GOLDEN))["cases"]
    for c in mk.CASES:
        assert mk.case_digest(c) == stored[c["name"]]["sha256_16"], c["name"]
