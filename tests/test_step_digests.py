"""Output digests of the M = 1 Llama-3-8B-shaped step against tests/golden/m1_step_digests.json.

The golden digests were written by tests/golden/make_step_digests.py, which calls only the oracle
and the seeded input generator.  The CPU test re-derives them (the oracle and the generator have
not drifted); the GPU test hashes rg_linear's outputs on the same inputs and needs no oracle run:
the same bytes on every run and every device that follows the order.
"""
import json
import os

import numpy as np
import pytest

from tests.golden import make_step_digests as mk

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "m1_step_digests.json")


def _golden():
    return json.load(open(GOLDEN))["layers"]


def test_oracle_reproduces_the_stored_step_digests():
    got = mk.step_digests()
    want = _golden()
    assert {n: d["sha256_16"] for n, d in got.items()} == {n: d["sha256_16"] for n, d in want.items()}


@pytest.mark.gpu
def test_gpu_step_outputs_match_the_stored_digests():
    import torch
    import synth
    import paper_2609_25624_amd as rg
    from tests import gpu_util as gu
    want = _golden()
    for li, (name, N, K) in enumerate(mk.LAYERS):
        assert want[name]["layer"] == li and (want[name]["N"], want[name]["K"]) == (N, K)
        gu.log(f"digest {name} ({N}x{K})")
        x, w = synth.layer_inputs(1, N, K, seed=0, w_std=0.02, layer=li)
        xd = torch.from_numpy(x).to(gu.dev())
        wd = torch.from_numpy(w.view(np.int16)).to(gu.dev())
        y = torch.empty((1, N), dtype=torch.float32, device=gu.dev())
        for _ in range(3):                      # repeated calls give the same bytes
            rg.rg_linear(xd, wd, y)
            torch.cuda.synchronize()
            assert mk.digest(y.cpu().numpy()) == want[name]["sha256_16"], name
