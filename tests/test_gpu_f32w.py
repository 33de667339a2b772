"""FP32 weights on the GPU (rg_linear_f32w) against the CPU oracle, bit for bit.

The paper's determinism probes use BF16 and FP32 weights alike (Supplement C);
the order is the same, with each weight used as the float32 it is.  Covered:
every kernel the FP32-weight planner can pick (the streaming kernel for M <= 4,
ktile, tiled, generic), ragged N and K, the hand-derived FP32-weight probes,
launch settings, and agreement with rg_linear when the weights are widened
BF16 values.
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


def _inputs(M, N, K, seed, std=0.02):
    x = synth.normal_f32(M, K, seed, 1, 1.0)
    w = synth.normal_f32(N, K, seed, 5, std)      # full-precision float32 weights
    return x, w


def _run(x, w):
    import torch
    import paper_2609_25624_amd as rg
    xd = torch.from_numpy(np.ascontiguousarray(x)).to(gu.dev())
    wd = torch.from_numpy(np.ascontiguousarray(w)).to(gu.dev())
    y = torch.empty((x.shape[0], w.shape[0]), dtype=torch.float32, device=gu.dev())
    rg.rg_linear_f32w(xd, wd, y)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def _check(M, N, K, seed=0, kernel=None, **launch):
    import oracle
    import paper_2609_25624_amd as rg
    if kernel or launch:
        rg.rg_linear_set_launch(kernel=kernel or 0, **launch) if kernel else rg.rg_linear_set_launch(**launch)
    plan = rg.rg_plan_f32w(M, N, K)
    if kernel:
        assert plan["kernel_name"] == kernel
    gu.log(f"f32w ({M},{N},{K}) seed={seed} -> {plan['kernel_name']} grid={plan['grid_wgs']} {launch}")
    x, w = _inputs(M, N, K, seed)
    gu.assert_bitwise(_run(x, w), oracle.linear_f32w(x, w), f"f32w ({M},{N},{K}) {plan['kernel_name']} {launch}")


@pytest.mark.parametrize("M", [1, 2, 3, 4])
@pytest.mark.parametrize("N,K", [(1, 4), (7, 252), (8, 256), (9, 260), (1030, 1000), (515, 4096), (64, 4100),
                                 (33, 14336)])
def test_stream_kernel_shapes(M, N, K):
    _check(M, N, K, seed=M + N + K, kernel="stream")


@pytest.mark.parametrize("M,N,K", [(5, 300, 1000), (16, 1030, 4096), (33, 257, 2052), (64, 100, 520)])
def test_ktile_with_fp32_weights(M, N, K):
    _check(M, N, K, seed=3, kernel="ktile")


@pytest.mark.parametrize("M,N,K", [(65, 130, 1000), (100, 257, 4100), (128, 256, 264)])
def test_tiled_with_fp32_weights(M, N, K):
    _check(M, N, K, seed=4, kernel="tiled")


@pytest.mark.parametrize("M,N,K", [(1, 10, 7), (3, 33, 1001), (70, 20, 259)])
def test_generic_with_fp32_weights(M, N, K):
    _check(M, N, K, seed=5)          # K % 4 != 0: the planner's generic kernel


@pytest.mark.parametrize("launch", [dict(grid_wgs=1), dict(grid_wgs=7, grid_order=1), dict(grid_wgs=3000),
                                    dict(grid_order=1)])
def test_stream_kernel_launch_settings(launch):
    _check(2, 1030, 4352, seed=9, kernel="stream", **launch)


def test_fp32_weight_probes_on_gpu():
    from tests import oracle_pins as pins
    for p in pins.load_f32w_probes():
        x, w = pins.f32w_probe_inputs(p)
        got = gu.bits(_run(x, w))[0, 0]
        assert got == int(p["expect_bits"], 16), (p["name"], hex(got))


@pytest.mark.parametrize("name,N,K", [("qkv", 6144, 4096), ("down", 4096, 14336)])
@pytest.mark.parametrize("M", [1, 4])
def test_widened_bf16_weights_match_rg_linear(name, N, K, M):
    # Same order, same values: FP32 weights that hold widened BF16 weights give rg_linear's bits.
    import torch
    x, wb = gu.layer(M, N, K, seed=11)
    xd, wd = gu.to_dev(x, wb)
    y16 = gu.run(xd, wd)
    torch.cuda.synchronize()
    w32 = (wb.astype(np.uint32) << 16).view(np.float32)
    gu.assert_bitwise(_run(x, w32), y16.cpu().numpy(), f"{name} M={M} widened BF16 as FP32")
    gu.assert_bitwise(y16.cpu().numpy(), gu.oracle_full(x, wb), f"{name} M={M} rg_linear")


def test_llama_down_m1_full_size():
    _check(1, 4096, 14336, seed=12)
