"""Signed zeros through every kernel, bit for bit against the oracle.

A row whose every 256-segment chain ends at -0 (each segment opens with a
negative product below half the smallest subnormal, probe O8, and continues
with -0 * 1.0 terms) must give y = -0 wherever the library places it: in the
register-tiled prefill kernel with a short last slab (K % 16 = 8, staged as
padding), in both 128 x 128 builds, and in every other kernel.  The same for
attention: a value numerator that is -0 must stay -0 through the positions
past the sequence.  (Design, R1: the result is the IEEE-754 one, signs of
zero included.)
"""
import numpy as np
import pytest

from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

NEG0 = 0x80000000


@pytest.fixture(autouse=True)
def _reset_launch():
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(None)
    yield
    rg.rg_linear_set_launch(None)


def _plant(x, w, rows, cols):
    """x rows `rows` and W rows `cols` become the all-segments -0 pattern."""
    K = x.shape[1]
    for m in rows:
        x[m] = -0.0
        x[m, 0::256] = -(2.0 ** -100)
    for n in cols:
        w[n] = 0x3F80
        w[n, 0::256] = 0x2180


def _check_planted(M, N, K, rows, cols, full=True, seed=0):
    import torch
    import oracle
    x, w = gu.layer(M, N, K, seed=seed)
    x, w = x.copy(), w.copy()
    _plant(x, w, rows, cols)
    xd, wd = gu.to_dev(x, w)
    y = gu.run(xd, wd)
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    rr = np.array([m for m in rows for _ in cols], dtype=np.int64)
    cc = np.array([n for _ in rows for n in cols], dtype=np.int64)
    want_pts = oracle.linear_sampled(x, w, rr, cc)
    assert np.all(gu.bits(want_pts) == NEG0)
    gu.assert_bitwise(got[rr, cc], want_pts, f"({M},{N},{K}) planted -0 outputs")
    if full:
        gu.assert_bitwise(got, gu.oracle_full(x, w), f"({M},{N},{K}) with -0 rows")
    else:
        # whole planted rows and columns
        rr = np.concatenate([np.repeat(rows, N), np.tile(np.arange(M), len(cols))])
        cc = np.concatenate([np.tile(np.arange(N), len(rows)), np.repeat(cols, M)])
        gu.assert_bitwise(got[rr, cc], oracle.linear_sampled(x, w, rr, cc), f"({M},{N},{K}) planted rows/cols")


@pytest.mark.parametrize("K", [8, 264, 1000])
def test_tiled_short_last_slab_keeps_minus_zero(K):
    import paper_2609_25624_amd as rg
    M, N = 65, 130
    assert rg.rg_plan(M, N, K)["kernel_name"] == "tiled"
    _check_planted(M, N, K, rows=[0, 33, 64], cols=[0, 77, 129], seed=K)


@pytest.mark.parametrize("K", [8, 264, 1000])
@pytest.mark.parametrize("depth", [2, 3])
def test_tiled_128_builds_keep_minus_zero(K, depth):
    import paper_2609_25624_amd as rg
    M, N = 2048, 4100
    rg.rg_linear_set_launch(kernel="tiled", depth=depth)
    p = rg.rg_plan(M, N, K)
    assert (p["kernel_name"], p["tile_m"], p["depth"]) == ("tiled", 128, depth)
    _check_planted(M, N, K, rows=[0, 1000, 2047], cols=[0, 2050, 4099], full=(K == 8), seed=K + depth)


def _kernel_cases():
    # (kernel, M, N, K) valid for each forced kernel; K ragged where the kernel allows it
    return [
        ("generic", 3, 40, 300), ("generic", 2, 33, 7),
        ("decode_xs", 1, 1030, 4352), ("decode", 1, 1030, 1000), ("decode", 2, 515, 14336),
        ("decode", 4, 300, 520),
        ("gemv", 1, 1030, 4096), ("gemv", 1, 515, 8192),
        ("ktile", 5, 130, 1000), ("ktile", 16, 301, 4104), ("ktile", 64, 77, 520),
        ("stream", 1, 33, 264), ("stream", 4, 130, 4352),
        ("tiled", 100, 1000, 1000), ("tiled", 129, 257, 264),
        ("skinny", 2, 33, 264), ("skinny", 4, 1030, 4104), ("skinny", 9, 77, 1000), ("skinny", 16, 130, 4096),
        ("wtile", 64, 130, 1000), ("wtile", 40, 77, 264), ("wtile", 65, 70, 8),
    ]


@pytest.mark.parametrize("kernel,M,N,K", _kernel_cases())
def test_every_kernel_keeps_minus_zero(kernel, M, N, K):
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(kernel=kernel)
    assert rg.rg_plan(M, N, K)["kernel_name"] == kernel
    rows = sorted({0, M - 1})
    cols = sorted({0, N // 2, N - 1})
    _check_planted(M, N, K, rows=rows, cols=cols, seed=M + N + K)


def _attn_dev(*arrs):
    import torch
    out = []
    for a in arrs:
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            a = a.view(np.int16)
        out.append(torch.from_numpy(a.copy()).to(gu.dev()))
    return out


@pytest.mark.parametrize("D", [64, 96, 128, 200, 256])
@pytest.mark.parametrize("G", [1, 3])
def test_attention_minus_zero_numerators(D, G):
    """Every segment's numerators end at -0: its first position has a tiny weight
    e = EXP1(-20) and value -2^-133 (their product rounds to -0), every other value is -0;
    the row maximum sits at position 1 (score 0).  Lengths 2 (one short segment) and 259
    (a second segment of three positions) leave most positions of the last segment past
    the sequence, where the kernels pad."""
    import torch
    import oracle
    import paper_2609_25624_amd as rg
    B, Hkv, Lmax = 2, 2, 300
    H = G * Hkv
    lens = np.array([2, 259], np.int32)
    q = np.zeros((B, H, D), np.float32)
    q[:, :, 0] = 1.0
    kc = np.zeros((B, Hkv, Lmax, D), np.uint16)
    vc = np.full((B, Hkv, Lmax, D), 0x8000, np.uint16)        # -0
    for l0 in (0, 256):
        kc[:, :, l0, 0] = 0xC1A0                               # bf16 -20.0: score -20
        vc[:, :, l0, :] = 0x8001                               # -2^-133
    want = oracle.attn_decode(q, kc, vc, lens, np.float32(1.0))
    assert np.all(gu.bits(want) == NEG0)
    qd, kd, vd, ld = _attn_dev(q, kc, vc, lens)
    out = torch.empty(qd.shape, dtype=torch.float32, device=gu.dev())
    rg.rg_attn_decode(qd, kd, vd, ld, out, 1.0)
    torch.cuda.synchronize()
    gu.assert_bitwise(out.cpu().numpy(), want, f"attention -0 numerators D={D} G={G}")
