"""The skinny kernel (M <= 16, and to M = 64 on narrow layers: 16 W rows x 4 segments per wave, x shared by the 16 lanes of a
DPP row) against the oracle, bit for bit.

Shapes cover the batched-decode layers of an 8B Llama-3-class model (Supplement A, decode
latency; Design, the decode bucket of R4), ragged row groups (N % 16 != 0), short last
segments (K % 256 != 0), segment counts that leave rows of a wave idle (J % 4 != 0), several
segment groups per wave (J > 32), slices of x (M > 8, or x registers capped), every build
(rows of x per slice 1, 2, 4, 8; segment groups per wave 1, 2, 4; depth 2, 3) and the
launch overrides.
"""
import numpy as np
import pytest

from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _reset_launch():
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(None)
    yield
    rg.rg_linear_set_launch(None)


def _check(M, N, K, seed=0, cfg=None, expect=None, bias=False):
    import torch
    import oracle
    import paper_2609_25624_amd as rg
    if cfg is not None:
        rg.rg_linear_set_launch(kernel="skinny", **cfg)
    p = rg.rg_plan(M, N, K)
    assert p["kernel_name"] == "skinny", p
    if expect:
        for k, v in expect.items():
            assert p[k] == v, (k, p)
    gu.log(f"skinny M={M} N={N} K={K} seed={seed} cfg={cfg} nw={p['waves_per_wg']} "
           f"grid={p['grid_wgs']} depth={p['depth']} mt={p['tile_m']}")
    x, w = gu.layer(M, N, K, seed=seed)
    xd, wd = gu.to_dev(x, w)
    if bias:
        b = np.random.default_rng(seed).standard_normal(N).astype(np.float32)
        bd = torch.from_numpy(b).to(gu.dev())
        y = torch.empty((M, N), dtype=torch.float32, device=gu.dev())
        rg.rg_linear_bias(xd, wd, bd, y)
        torch.cuda.synchronize()
        gu.assert_bitwise(y.cpu().numpy(), oracle.linear_bias(x, w, b), f"skinny bias ({M},{N},{K})")
        return
    y = gu.run(xd, wd)
    torch.cuda.synchronize()
    gu.assert_bitwise(y.cpu().numpy(), gu.oracle_full(x, w), f"skinny ({M},{N},{K}) {cfg}")


@pytest.mark.parametrize("M", [1, 2, 3, 4, 8, 16])
@pytest.mark.parametrize("N,K", [(6144, 4096), (4096, 4096), (28672, 4096), (4096, 14336)])
def test_llama_decode_layers_full_output(M, N, K):
    # (the planner gives M = 1 on 4096 x 4096 to the GEMV; the skinny kernel is forced there)
    _check(M, N, K, seed=M * 7 + K, cfg={} if M == 1 else None)


@pytest.mark.parametrize("M", [1, 2, 4, 5, 9, 16])
@pytest.mark.parametrize("N,K", [(1, 8), (15, 264), (17, 1000), (33, 1280), (130, 2056), (1000, 4104),
                                 (77, 9000), (31, 14336), (19, 28672)])
def test_ragged_shapes(M, N, K):
    _check(M, N, K, seed=M + N + K)


@pytest.mark.parametrize("M", [17, 24, 33, 64])
@pytest.mark.parametrize("N,K", [(4096, 4096), (259, 14336), (1030, 2056)])
def test_mid_batch_narrow_layers(M, N, K):
    """16 < M <= 64 on layers with few 64-row tiles: the planner's skinny kernel, several
    slices of x with a short last one."""
    _check(M, N, K, seed=M * 3 + N)


@pytest.mark.parametrize("M,N,K,sm,mt,nw", [
    (2, 300, 4096, 2, 2, 4),      # one segment group per wave
    (2, 300, 9000, 2, 2, 5),      # two per wave (J = 36)
    (2, 100, 28672, 2, 2, 7),     # four per wave (J = 112)
    (4, 300, 4096, 4, 4, 4),
    (4, 300, 14336, 4, 4, 7),     # two per wave
    (8, 300, 4096, 8, 8, 4),
    (8, 300, 14336, 8, 4, 7),     # x registers cap the slice at 4 rows: two slices
    (16, 300, 28672, 2, 2, 7),    # eight slices of 2 rows
    (16, 300, 4096, 0, 1, 4),     # the planner's narrowest slices: sixteen of one row
    (3, 6144, 4096, 0, 2, 4),     # planner: two slices of 2 rows (more workgroups)
    (8, 4096, 4096, 0, 4, 4),     # planner: two slices of 4 rows
])
def test_every_build(M, N, K, sm, mt, nw):
    _check(M, N, K, seed=N + K, cfg=dict(slice_m=sm) if sm else None, expect={"tile_m": mt, "waves_per_wg": nw})


@pytest.mark.parametrize("cfg", [dict(depth=2), dict(depth=3), dict(depth=2, grid_order=1), dict(grid_wgs=1),
                                 dict(grid_wgs=3, depth=3), dict(grid_wgs=1000, grid_order=1),
                                 dict(waves_per_wg=8), dict(waves_per_wg=2, depth=2), dict(waves_per_wg=1, grid_wgs=7),
                                 dict(slice_m=1), dict(slice_m=2, depth=3), dict(slice_m=8, grid_wgs=5)])
@pytest.mark.parametrize("M,N,K", [(4, 1030, 4096), (3, 515, 2056), (16, 259, 4352)])
def test_launch_overrides_do_not_change_bits(M, N, K, cfg):
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(kernel="skinny", **cfg)
    try:
        rg.rg_plan(M, N, K)
    except rg.RgError:
        pytest.skip(f"{cfg} not valid for ({M},{N},{K})")
    _check(M, N, K, seed=5, cfg=cfg)


@pytest.mark.parametrize("M,N,K", [(4, 1030, 4096), (5, 77, 1000), (16, 301, 14336)])
def test_bias(M, N, K):
    _check(M, N, K, seed=9, bias=True)


def test_order_probes_inside_rows():
    """The hand-derived probes placed at x row 5 of a 9-row batch (second slice) and spread
    over W rows of a 1030-row layer run through the skinny kernel."""
    import torch
    import oracle
    import paper_2609_25624_amd as rg
    from tests import oracle_pins as pins
    for i, p in enumerate(pins.load_probes()):
        x1, w1 = pins.probe_inputs(p)
        K = max(8, (x1.shape[1] + 7) // 8 * 8)
        X, W = gu.layer(9, 1030, K, seed=31 + i)
        X = X.copy(); W = W.copy()
        X[5] = 0.0
        X[5, :x1.shape[1]] = x1[0]
        row = 3 + 97 * i
        W[row] = 0
        W[row, :w1.shape[1]] = w1[0]
        assert rg.rg_plan(9, 1030, K)["kernel_name"] == "skinny"
        xd, wd = gu.to_dev(X, W)
        y = gu.run(xd, wd)
        torch.cuda.synchronize()
        got = y.cpu().numpy()
        gu.assert_bitwise(got, gu.oracle_full(X, W), f"probe {p['name']} batch")
        if x1.shape[1] == K:
            want = int(p["expect_bits"], 16)
            assert int(gu.bits(got)[5, row]) == want, p["name"]


@pytest.mark.parametrize("N,K", [(6144, 4096), (4096, 14336), (33, 1280), (17, 1000), (1, 8), (130, 2056)])
@pytest.mark.parametrize("cfg", [dict(), dict(waves_per_wg=4), dict(depth=3, grid_order=1)])
def test_one_row_build_overrides(N, K, cfg):
    """M = 1 through the skinny kernel's one-row build, under launch overrides."""
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(kernel="skinny", **cfg)
    try:
        rg.rg_plan(1, N, K)
    except rg.RgError:
        pytest.skip(f"{cfg} not valid for (1,{N},{K})")
    _check(1, N, K, seed=N + K, cfg=cfg, expect={"tile_m": 1})
