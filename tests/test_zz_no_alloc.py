"""rg_attn_decode_noalloc (static device scratch, no allocation) against rg_attn_decode.

Two calls in a row through the C-ABI, the second with a smaller input, each compared
bit for bit with the entry point that takes a caller workspace and with the oracle;
then a workspace beyond the scratch is refused with RG_ERR_RANGE.
"""
import numpy as np
import pytest

import synth
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


def _dev(*arrs):
    import torch
    out = []
    for a in arrs:
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            a = a.view(np.int16)
        out.append(torch.from_numpy(a.copy()).to(gu.dev()))
    return out


def _same(got, want, what):
    g, w = gu.bits(got), gu.bits(want)
    nan = np.isnan(got) & np.isnan(want)
    assert np.array_equal(np.isnan(got), np.isnan(want)), what
    bad = np.flatnonzero(~((g == w) | nan).ravel())
    assert bad.size == 0, f"{what}: {bad.size} differ, first flat {bad[0]}"


def _case(B, H, Hkv, Lmax, D, lens, seed):
    import torch
    import oracle
    import paper_2609_25624_amd as rg
    gu.log(f"noalloc B={B} H={H} Hkv={Hkv} Lmax={Lmax} D={D} lens={list(lens)[:4]}")
    q, kc, vc = synth.attn_inputs(B, H, Hkv, Lmax, D, seed=seed)
    scale = np.float32(1.0 / np.sqrt(D))
    qd, kd, vd, ld = _dev(q, kc, vc, np.asarray(lens, np.int32))
    out_ws = torch.full(qd.shape, float("nan"), dtype=torch.float32, device=gu.dev())
    out_na = torch.full(qd.shape, float("nan"), dtype=torch.float32, device=gu.dev())
    rg.rg_attn_decode(qd, kd, vd, ld, out_ws, scale)
    rg.rg_attn_decode_noalloc(qd, kd, vd, ld, out_na, scale)
    torch.cuda.synchronize()
    a, b = out_ws.cpu().numpy(), out_na.cpu().numpy()
    _same(b, a, "noalloc vs workspace entry point")
    _same(b, oracle.attn_decode(q, kc, vc, lens, scale), "noalloc vs oracle")


def test_noalloc_matches_workspace_entry_point_twice_then_smaller():
    _case(8, 32, 8, 2048, 128, [2048, 1500, 7, 1025, 1, 256, 257, 2000], seed=71)
    _case(2, 6, 3, 300, 64, [300, 41], seed=72)          # smaller: stale scratch contents are not read


def test_noalloc_refuses_workspace_beyond_scratch():
    import torch
    import paper_2609_25624_amd as rg
    B, H, Hkv, Lmax, D = 1, 8, 1, 2_200_000, 8
    assert rg.rg_attn_workspace_size(B, H, Lmax, D) > rg.ATTN_SCRATCH_BYTES
    q = torch.zeros((B, H, D), dtype=torch.float32, device=gu.dev())
    kc = torch.zeros((B, Hkv, Lmax, D), dtype=torch.int16, device=gu.dev())
    lens = torch.ones(B, dtype=torch.int32, device=gu.dev())
    out = torch.full_like(q, 7.0)
    with pytest.raises(rg.RgError) as e:
        rg.rg_attn_decode_noalloc(q, kc, kc.clone(), lens, out, 1.0)
    assert e.value.code == rg.RG_ERR_RANGE
    torch.cuda.synchronize()
    assert torch.all(out == 7.0).item()                  # nothing was enqueued
