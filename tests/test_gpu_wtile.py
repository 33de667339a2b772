"""The wave-tile kernel (64 x 64 output tiles; each wave the whole tile for one segment at a
time, 8 x 8 chains per lane, the partials added wave by wave in segment order) against the
oracle, bit for bit.

Shapes: the wide decode layers it serves (gate+up of an 8B Llama-3-class model, the LM head,
the 70B gate+up; Design, the decode bucket of R4), ragged tiles in M and N, short last
segments and slabs (K % 256 != 0, K % 16 == 8), fewer segments than waves (J < 4), several
rounds (J > 4, J % 4 != 0), more than one row of tiles (M > 64, forced), the bias, FP32
weights, the reversed grid order and rows that must stay -0.
"""
import numpy as np
import pytest

import synth
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _reset_launch():
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(None)
    yield
    rg.rg_linear_set_launch(None)


def _check(M, N, K, seed=0, forced=True, bias=False, **launch):
    import torch
    import oracle
    import paper_2609_25624_amd as rg
    if forced:
        rg.rg_linear_set_launch(kernel="wtile", **launch)
    p = rg.rg_plan(M, N, K)
    assert p["kernel_name"] == "wtile", p
    gu.log(f"wtile M={M} N={N} K={K} seed={seed} grid={p['grid_wgs']} {launch} bias={bias}")
    x, w = gu.layer(M, N, K, seed=seed)
    xd, wd = gu.to_dev(x, w)
    if bias:
        b = np.random.default_rng(seed).standard_normal(N).astype(np.float32)
        y = torch.empty((M, N), dtype=torch.float32, device=gu.dev())
        rg.rg_linear_bias(xd, wd, torch.from_numpy(b).to(gu.dev()), y)
        torch.cuda.synchronize()
        gu.assert_bitwise(y.cpu().numpy(), oracle.linear_bias(x, w, b), f"wtile bias ({M},{N},{K})")
        return
    y = gu.run(xd, wd)
    torch.cuda.synchronize()
    gu.assert_bitwise(y.cpu().numpy(), gu.oracle_full(x, w), f"wtile ({M},{N},{K}) {launch}")


@pytest.mark.parametrize("M", [33, 48, 64])
def test_gate_up_layer_full_output(M):
    _check(M, 28672, 4096, seed=M)


@pytest.mark.parametrize("M,N,K", [(64, 4096, 14336), (40, 1030, 8192), (64, 57344 // 8, 8192)])
def test_long_k_layers(M, N, K):
    _check(M, N, K, seed=N + K)


@pytest.mark.parametrize("M,N,K", [(1, 1, 8), (5, 77, 1000), (33, 130, 2056), (64, 100, 264), (63, 65, 520),
                                   (64, 64, 256), (17, 200, 768), (64, 129, 1288), (65, 70, 520), (130, 300, 4104)])
def test_ragged_shapes(M, N, K):
    _check(M, N, K, seed=M * 7 + N + K)


@pytest.mark.parametrize("M,N,K", [(64, 1030, 4096), (40, 77, 1000), (65, 70, 520), (5, 33, 264), (64, 200, 14336),
                                   (64, 130, 2304)])
def test_eight_wave_build(M, N, K):
    _check(M, N, K, seed=M + N, waves_per_wg=8)


@pytest.mark.parametrize("M,N,K", [(64, 1030, 4096), (40, 77, 1000)])
def test_bias(M, N, K):
    _check(M, N, K, seed=11, bias=True)


@pytest.mark.parametrize("M,N,K", [(64, 1030, 4096), (37, 130, 264)])
def test_reversed_grid_order(M, N, K):
    _check(M, N, K, seed=13, grid_order=1)


@pytest.mark.parametrize("M,N,K", [(48, 1030, 4096), (64, 77, 1000), (9, 33, 264)])
def test_fp32_weights(M, N, K):
    import torch
    import oracle
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(kernel="wtile")
    assert rg.rg_plan_f32w(M, N, K)["kernel_name"] == "wtile"
    x = synth.normal_f32(M, K, M + N, 1, 1.0)
    w = synth.normal_f32(N, K, M + N, 5, 0.02)
    xd = torch.from_numpy(np.ascontiguousarray(x)).to(gu.dev())
    wd = torch.from_numpy(np.ascontiguousarray(w)).to(gu.dev())
    y = torch.empty((M, N), dtype=torch.float32, device=gu.dev())
    rg.rg_linear_f32w(xd, wd, y)
    torch.cuda.synchronize()
    gu.assert_bitwise(y.cpu().numpy(), oracle.linear_f32w(x, w), f"wtile f32w ({M},{N},{K})")


def test_launch_overrides_rejected_or_neutral():
    import paper_2609_25624_amd as rg
    for bad in (dict(waves_per_wg=2), dict(grid_wgs=100), dict(depth=2), dict(tile_n=32), dict(slice_m=2)):
        rg.rg_linear_set_launch(kernel="wtile", **bad)
        with pytest.raises(rg.RgError):
            rg.rg_plan(64, 4096, 4096)
    rg.rg_linear_set_launch(None)
    _check(64, 1030, 4096, seed=17, waves_per_wg=4, tile_n=64)


def test_order_probes_inside_tiles():
    """The hand-derived order probes placed at x row 37 and spread over W rows of a 1030-row
    layer, through the wave-tile kernel."""
    import torch
    import paper_2609_25624_amd as rg
    from tests import oracle_pins as pins
    rg.rg_linear_set_launch(kernel="wtile")
    for i, p in enumerate(pins.load_probes()):
        x1, w1 = pins.probe_inputs(p)
        K = max(8, (x1.shape[1] + 7) // 8 * 8)
        X, W = gu.layer(48, 1030, K, seed=41 + i)
        X = X.copy(); W = W.copy()
        X[37] = 0.0
        X[37, :x1.shape[1]] = x1[0]
        row = 5 + 97 * i
        W[row] = 0
        W[row, :w1.shape[1]] = w1[0]
        assert rg.rg_plan(48, 1030, K)["kernel_name"] == "wtile"
        xd, wd = gu.to_dev(X, W)
        y = gu.run(xd, wd)
        torch.cuda.synchronize()
        got = y.cpu().numpy()
        gu.assert_bitwise(got, gu.oracle_full(X, W), f"probe {p['name']} in a wave tile")
        if x1.shape[1] == K:
            assert int(gu.bits(got)[37, row]) == int(p["expect_bits"], 16), p["name"]
