"""Weights (and attention caches) beyond 4 GiB: 64-bit addressing in every kernel family.

W is a seeded block of R = 1021 rows repeated down N rows on the GPU, so every output
must equal the oracle's output for row n mod R.  The shapes put rows past the 4 GiB
mark: for K = 2304, 2^32 bytes is not a whole number of rows, and for K = 4096 it is
524288 rows, which is not a multiple of R.  A 32-bit offset that wrapped would read
other weights and change the bits.  Every output is compared, not a sample.
"""
import numpy as np
import pytest

from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

_R = 1021


@pytest.fixture(autouse=True)
def _reset_launch():
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(None)
    yield
    rg.rg_linear_set_launch(None)


@pytest.mark.parametrize("M,N,K,kernel,forced", [(1, 1048579, 2304, "skinny", False), (1, 524309, 4096, "skinny", False),
                                                 (1, 1048579, 2304, "decode_xs", True), (1, 524309, 4096, "gemv", True),
                                                 (3, 1048579, 2304, "skinny", False), (16, 1048579, 2304, "skinny", False),
                                                 (3, 1048579, 2304, "decode", True), (16, 1048579, 2304, "ktile", True),
                                                 (40, 1048579, 2304, "wtile", True), (40, 1048579, 2304, "skinny", True),
                                                 (70, 1048579, 2304, "tiled", False)])
def test_weights_beyond_4_gib(M, N, K, kernel, forced):
    import torch
    import paper_2609_25624_amd as rg
    assert 2 * N * K > (1 << 32)
    rg.rg_linear_set_launch(kernel=kernel) if forced else rg.rg_linear_set_launch(None)
    plan = rg.rg_plan(M, N, K)
    assert plan["kernel_name"] == kernel
    gu.log(f"large W: M={M} N={N} K={K} ({2 * N * K / 2**30:.2f} GiB) kernel={kernel}")
    x, wblock = gu.layer(M, _R, K, seed=77 + M)
    want_block = gu.oracle_full(x, wblock)
    xd, wb = gu.to_dev(x, wblock)
    reps = (N + _R - 1) // _R
    wbig = wb.repeat(reps, 1)[:N]
    assert wbig.is_contiguous() and wbig.shape == (N, K)
    y = torch.empty((M, N), dtype=torch.float32, device=gu.dev())
    rg.rg_linear(xd, wbig, y)
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    del wbig, y
    torch.cuda.empty_cache()
    want = np.tile(want_block, (1, reps))[:, :N]
    gu.assert_bitwise(got, want, f"large W ({M},{N},{K}) {kernel}")


def test_attention_caches_beyond_4_gib():
    """Two sequences in 4.3 GB key and value caches, the second one's elements at offsets past
    2^31: its output must equal the same sequence alone in a fresh cache at offset 0 (the order
    does not depend on the batch or on where a sequence sits), and the first sequence's output
    must equal the oracle.  The caches repeat a seeded 4099-position block along the sequence."""
    import torch
    import oracle
    import synth
    import paper_2609_25624_amd as rg
    B, H, Hkv, D, P = 2, 2, 1, 256, 4099
    Lmax = (1 << 22) + 4097
    assert Lmax * D > (1 << 30) and B * Hkv * Lmax * D * 2 > (1 << 32)
    gu.log(f"large attention: B={B} Lmax={Lmax} D={D} ({B * Hkv * Lmax * D * 2 / 2**30:.2f} GiB per cache)")
    q, kb, vb = synth.attn_inputs(B, H, Hkv, P, D, seed=91)
    reps = (Lmax + P - 1) // P
    kbd = torch.from_numpy(kb.view(np.int16).copy()).to(gu.dev())
    vbd = torch.from_numpy(vb.view(np.int16).copy()).to(gu.dev())
    kd = kbd.repeat(1, 1, reps, 1)[:, :, :Lmax].contiguous()
    vd = vbd.repeat(1, 1, reps, 1)[:, :, :Lmax].contiguous()
    qd = torch.from_numpy(q.copy()).to(gu.dev())
    scale = np.float32(1.0 / np.sqrt(D))
    lens = np.array([P - 3, Lmax - 5], np.int32)
    out = torch.empty((B, H, D), dtype=torch.float32, device=gu.dev())
    rg.rg_attn_decode(qd, kd, vd, torch.from_numpy(lens.copy()).to(gu.dev()), out, scale)
    # the second sequence alone, at offset 0
    k1 = kd[1:2].clone()
    v1 = vd[1:2].clone()
    out1 = torch.empty((1, H, D), dtype=torch.float32, device=gu.dev())
    rg.rg_attn_decode(qd[1:2].contiguous(), k1, v1, torch.from_numpy(lens[1:2].copy()).to(gu.dev()), out1, scale)
    torch.cuda.synchronize()
    got, alone = out.cpu().numpy(), out1.cpu().numpy()
    del kd, vd, k1, v1
    torch.cuda.empty_cache()
    assert np.array_equal(gu.bits(got[1]), gu.bits(alone[0])), "sequence past 2^31 elements vs alone"
    # the first sequence (its positions lie in the first block) against the oracle
    want0 = oracle.attn_decode(q[:1], kb[:1], vb[:1], lens[:1], scale)
    assert np.array_equal(gu.bits(got[:1]), gu.bits(want0)), "first sequence vs oracle"
