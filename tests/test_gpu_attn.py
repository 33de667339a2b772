"""Fixed-order decode attention (rg_attn_decode) on the GPU against the CPU oracle, bit for bit.

Shapes: grouped-query heads (1 to 8 query heads per kv head), head dims 8 to 256,
ragged lengths across the 256-position segments (including length 0, which
gives NaN by definition), the hand-derived probes, a Llama-3-8B-shaped decode
batch, and the invariants the order promises: a sequence's output does not
depend on the rest of the batch, on Lmax, on repeats or on the CU mask.
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


def _run(q, kc, vc, lens, scale, stream=None):
    import torch
    import paper_2609_25624_amd as rg
    qd, kd, vd, ld = _dev(q, kc, vc, np.asarray(lens, np.int32))
    out = torch.empty(qd.shape, dtype=torch.float32, device=gu.dev())
    rg.rg_attn_decode(qd, kd, vd, ld, out, scale, stream=stream)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def _assert_same(got, want, what):
    g, w = gu.bits(got), gu.bits(want)
    nan_g, nan_w = np.isnan(got), np.isnan(want)
    assert np.array_equal(nan_g, nan_w), f"{what}: NaN positions differ"
    ok = (g == w) | (nan_g & nan_w)          # NaN payloads of 0/0 differ between CPUs and GPUs
    if not ok.all():
        i = int(np.flatnonzero(~ok.ravel())[0])
        raise AssertionError(f"{what}: {int((~ok).sum())}/{ok.size} differ; first flat {i}: "
                             f"gpu 0x{g.ravel()[i]:08x} oracle 0x{w.ravel()[i]:08x}")


def _check(B, H, Hkv, Lmax, D, lens, seed=0, scale=None, kstd=1.0):
    import oracle
    gu.log(f"attn B={B} H={H} Hkv={Hkv} Lmax={Lmax} D={D} lens={list(lens)[:6]} seed={seed}")
    q, kc, vc = synth.attn_inputs(B, H, Hkv, Lmax, D, seed=seed, kstd=kstd)
    scale = np.float32(1.0 / np.sqrt(D)) if scale is None else np.float32(scale)
    got = _run(q, kc, vc, lens, scale)
    _assert_same(got, oracle.attn_decode(q, kc, vc, lens, scale), f"attn ({B},{H},{Hkv},{Lmax},{D})")
    return q, kc, vc, got


@pytest.mark.parametrize("H,Hkv", [(1, 1), (2, 1), (3, 1), (4, 2), (5, 1), (6, 3), (7, 7), (8, 1), (32, 8)])
def test_group_sizes(H, Hkv):
    _check(2, H, Hkv, 300, 64, [300, 41], seed=H * 10 + Hkv)


@pytest.mark.parametrize("H,Hkv", [(1, 1), (3, 1), (8, 1), (16, 2), (7, 7)])
@pytest.mark.parametrize("D", [128, 256])
def test_group_sizes_at_the_wide_head_dims(H, Hkv, D):
    """Group sizes at D = 128 and 256 (one wave per work item in the partials pass; the
    two-positions-per-thread scores kernel for eight heads per kv head), ragged lengths."""
    _check(3, H, Hkv, 600, D, [600, 257, 1], seed=H * 100 + Hkv + D)


@pytest.mark.parametrize("D", [8, 16, 64, 96, 128, 136, 200, 256])
def test_head_dims(D):
    _check(2, 4, 2, 520, D, [520, 257], seed=D, kstd=2.0)


@pytest.mark.parametrize("lens", [[1, 255, 256, 257], [0, 3, 512, 513], [1024, 1000, 2, 769]])
def test_ragged_lengths(lens):
    _check(4, 8, 2, 1024, 128, lens, seed=sum(lens))


def test_lengths_beyond_lmax_are_clamped():
    _check(3, 4, 4, 300, 64, [-5, 300, 10 ** 6], seed=9)


def test_llama3_8b_decode_batch():
    rng = np.random.default_rng(1)
    lens = rng.integers(1, 4097, 16)
    lens[0], lens[1] = 4096, 1
    _check(16, 32, 8, 4096, 128, lens, seed=2)


def test_attention_probes_on_gpu():
    from tests import attn_pins as pins
    for p in pins.load_probes():
        q, kc, vc, lens = pins.probe_inputs(p)
        out = _run(q, kc, vc, lens, 1.0)
        got = int(gu.bits(out)[0, 0, 0])
        assert got == int(p["expect_bits"], 16), (p["name"], hex(got))
        assert np.all(gu.bits(out)[0, 0, 1:] == 0), p["name"]


def test_sequence_alone_and_lmax_do_not_change_bits():
    B, H, Hkv, Lmax, D = 3, 8, 2, 700, 128
    lens = [700, 256, 513]
    q, kc, vc, out = _check(B, H, Hkv, Lmax, D, lens, seed=21)
    for b in range(B):
        o1 = _run(q[b:b + 1], kc[b:b + 1], vc[b:b + 1], lens[b:b + 1], np.float32(1 / np.sqrt(D)))
        _assert_same(o1[0], out[b], f"sequence {b} alone")
    # a larger Lmax (padding after every sequence's cache) gives the same bits
    pad = np.zeros((B, Hkv, 300, D), np.uint16)
    o2 = _run(q, np.concatenate([kc, pad + 0x7F00], 2), np.concatenate([vc, pad + 0x4F00], 2), lens,
              np.float32(1 / np.sqrt(D)))
    _assert_same(o2, out, "Lmax 1000")


def test_repeats_and_cu_masks_give_one_result():
    import torch
    import paper_2609_25624_amd as rg
    B, H, Hkv, Lmax, D = 4, 32, 8, 2048, 128
    lens = [2048, 1500, 7, 1025]
    q, kc, vc, out = _check(B, H, Hkv, Lmax, D, lens, seed=31)
    qd, kd, vd, ld = _dev(q, kc, vc, np.asarray(lens, np.int32))
    o = torch.empty(qd.shape, dtype=torch.float32, device=gu.dev())
    seen = set()
    for _ in range(20):
        rg.rg_attn_decode(qd, kd, vd, ld, o, np.float32(1 / np.sqrt(D)))
        torch.cuda.synchronize()
        seen.add(o.cpu().numpy().tobytes())
    assert len(seen) == 1 and next(iter(seen)) == out.tobytes()
    ncu = rg.rg_device_cu_count()
    nwords = (ncu + 31) // 32
    for name, mask in {"half": [0xFFFFFFFF if i < nwords // 2 else 0 for i in range(nwords)],
                       "alternate": [0x55555555] * nwords}.items():
        try:
            s = rg.rg_stream_create_cu_mask(mask)
        except rg.RgError as e:
            gu.log(f"  cu mask {name}: refused ({e})")
            continue
        try:
            ext = torch.cuda.ExternalStream(s)
            torch.cuda.synchronize()
            rg.rg_attn_decode(qd, kd, vd, ld, o, np.float32(1 / np.sqrt(D)), stream=ext)
            ext.synchronize()
            _assert_same(o.cpu().numpy(), out, f"cu mask {name}")
        finally:
            torch.cuda.synchronize()
            rg.rg_stream_destroy(s)


def test_argument_errors():
    import torch
    import paper_2609_25624_amd as rg
    q = torch.zeros((1, 3, 64), device=gu.dev())
    kc = torch.zeros((1, 2, 16, 64), dtype=torch.int16, device=gu.dev())
    lens = torch.ones(1, dtype=torch.int32, device=gu.dev())
    out = torch.empty_like(q)
    with pytest.raises(rg.RgError):                     # H % Hkv != 0
        rg.rg_attn_decode(q, kc, kc.clone(), lens, out, 1.0)
    q9 = torch.zeros((1, 9, 64), device=gu.dev())
    k1 = torch.zeros((1, 1, 16, 64), dtype=torch.int16, device=gu.dev())
    with pytest.raises(rg.RgError):                     # more than 8 query heads per kv head
        rg.rg_attn_decode(q9, k1, k1.clone(), lens, torch.empty_like(q9), 1.0)
    q2 = torch.zeros((1, 2, 64), device=gu.dev())
    ws = torch.empty(8, dtype=torch.uint8, device=gu.dev())
    with pytest.raises(rg.RgError):                     # workspace too small
        rg.rg_attn_decode(q2, kc, kc.clone(), lens, torch.empty_like(q2), 1.0, workspace=ws)


def test_both_row_maximum_paths():
    """More work items than the partials kernel has waves (16 per CU, so B x 8 kv heads x 32
    segments with B = CUs / 16 + 1): the row maxima come from the maximum kernel; the same
    sequences in a smaller batch take them inside the partials kernel.  Both equal the oracle."""
    import paper_2609_25624_amd as rg
    B = rg.rg_device_cu_count() // 16 + 1
    H, Hkv, Lmax, D = 32, 8, 8192, 128
    assert B * Hkv * (Lmax // 256) > 16 * rg.rg_device_cu_count()
    lens = [8192 - 397 * (b % 17) for b in range(B)]
    q, kc, vc, got = _check(B, H, Hkv, Lmax, D, lens, seed=23)
    got2 = _run(q[:3], kc[:3], vc[:3], lens[:3], np.float32(1.0 / np.sqrt(D)))
    _assert_same(got2, got[:3], "first three sequences alone")


@pytest.mark.parametrize("D", [128, 256])
def test_whole_and_split_value_columns(D):
    """More work items than four per CU: one wave takes all value columns of an item; the
    first three sequences alone (few items): two waves split each item's columns.  Both
    equal the oracle and each other."""
    import paper_2609_25624_amd as rg
    H, Hkv, Lmax = 4, 2, 1024
    B = 4 * rg.rg_device_cu_count() // (Hkv * (Lmax // 256)) + 1
    assert B * Hkv * (Lmax // 256) > 4 * rg.rg_device_cu_count()
    assert 3 * Hkv * (Lmax // 256) <= 4 * rg.rg_device_cu_count()
    lens = [1024 - 97 * (b % 11) for b in range(B)]
    q, kc, vc, got = _check(B, H, Hkv, Lmax, D, lens, seed=31 + D)
    got2 = _run(q[:3], kc[:3], vc[:3], lens[:3], np.float32(1.0 / np.sqrt(D)))
    _assert_same(got2, got[:3], "first three sequences alone")


@pytest.mark.parametrize("H,L", [(4, 33000), (3, 44000), (7, 19000)])
def test_in_kernel_maximum_beyond_512_segment_maxima(H, L):
    """One sequence long enough that its G x Jb segment maxima exceed the 512 a wave loads with
    its first step (G = 4, 3, 7 query heads per kv head), so the partials wave folds the rest
    in its tail loop.  One kv head: few work items, so the in-kernel maximum path is taken."""
    assert H * (-(-L // 256)) > 512
    _check(1, H, 1, L, 128, [L], seed=H * 7 + L)
