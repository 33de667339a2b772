"""Output digests of the M = 1 Llama-3-8B-shaped step (and of the fixed-order decode attention on
a Llama-3-8B-shaped batch) against tests/golden/m1_step_digests.json.

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


def test_oracle_reproduces_the_stored_attention_digest():
    want = json.load(open(GOLDEN))["attention"]
    assert {k: want[k] for k in mk.ATTN} == mk.ATTN
    assert mk.attn_digest()["sha256_16"] == want["sha256_16"]


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


@pytest.mark.gpu
def test_gpu_attention_output_matches_the_stored_digest():
    import torch
    import paper_2609_25624_amd as rg
    from tests import gpu_util as gu
    want = json.load(open(GOLDEN))["attention"]
    gu.log("digest attention (16 x 32 heads, 8 kv heads, D 128, Lmax 4096)")
    q, kc, vc, lens, scale = mk.attn_case()
    qd = torch.from_numpy(q.copy()).to(gu.dev())
    kd = torch.from_numpy(kc.view(np.int16).copy()).to(gu.dev())
    vd = torch.from_numpy(vc.view(np.int16).copy()).to(gu.dev())
    ld = torch.from_numpy(lens.copy()).to(gu.dev())
    out = torch.empty(q.shape, dtype=torch.float32, device=gu.dev())
    for _ in range(3):                          # repeated calls give the same bytes
        rg.rg_attn_decode(qd, kd, vd, ld, out, scale)
        torch.cuda.synchronize()
        assert mk.digest(out.cpu().numpy()) == want["sha256_16"]
