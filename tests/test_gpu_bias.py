"""The bias variant (Design, eq. 2 with its +b term) on the GPU, through the C-ABI.

rg_linear_bias must equal the CPU oracle's fold-then-add bit for bit under every
kernel and launch setting, equal rg_linear's output plus b (one binary32 add on
the host), carry the hand-derived bias probes, and reject a NULL or aliased bias.
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


def _bias_dev(b):
    import torch
    return torch.from_numpy(np.array(b, dtype=np.float32, copy=True)).to(gu.dev())


def _run_bias(xd, wd, bd):
    import torch
    import paper_2609_25624_amd as rg
    y = torch.empty((xd.shape[0], wd.shape[0]), dtype=torch.float32, device=xd.device)
    rg.rg_linear_bias(xd, wd, bd, y)
    torch.cuda.synchronize()
    return y.cpu().numpy()


_SETTINGS = [
    dict(),
    dict(kernel="generic"),
    dict(kernel="decode"),
    dict(kernel="decode_xs"),
    dict(kernel="gemv"),
    dict(kernel="gemv", waves_per_wg=1, grid_wgs=7, grid_order=1),
    dict(kernel="ktile"),
    dict(kernel="ktile", tile_n=64),
    dict(kernel="ktile", tile_n=16, waves_per_wg=8),
    dict(kernel="tiled"),
    dict(kernel="stream"),
]


@pytest.mark.parametrize("M,N,K", [(1, 1030, 4096), (1, 777, 4352), (3, 301, 1000), (4, 2048, 2560),
                                   (16, 1030, 4104), (70, 515, 1024), (1, 5, 7), (2, 9, 257)])
def test_bias_matches_oracle_under_every_kernel(M, N, K):
    import oracle
    import paper_2609_25624_amd as rg
    x, w = gu.layer(M, N, K, seed=31)
    b = synth.layer_bias(N, seed=31)
    xd, wd = gu.to_dev(x, w)
    bd = _bias_dev(b)
    want = oracle.linear_bias(x, w, b)
    plain = gu.oracle_full(x, w)
    # the oracle's bias output is the bias-free product plus b, one binary32 add each
    gu.assert_bitwise(want, plain + b[None, :], "oracle bias = product + b")
    for cfg in _SETTINGS:
        rg.rg_linear_set_launch(**cfg) if cfg else rg.rg_linear_set_launch(None)
        try:
            plan = rg.rg_plan(M, N, K)
        except rg.RgError:
            continue                                # setting not valid for this shape
        gu.log(f"bias ({M},{N},{K}) launch {cfg} -> {plan['kernel_name']}")
        gu.assert_bitwise(_run_bias(xd, wd, bd), want, f"bias ({M},{N},{K}) launch {cfg}")
    rg.rg_linear_set_launch(None)


def test_bias_on_8b_gate_up_m1_and_m16():
    import oracle
    for M in (1, 16):
        N, K = 28672, 4096
        gu.log(f"bias gate_up M={M}")
        x, w = gu.layer(M, N, K, seed=5, layer_id=2)
        b = synth.layer_bias(N, seed=5, layer=2)
        got = _run_bias(*gu.to_dev(x, w), _bias_dev(b))
        rows, cols = gu.sample_indices(M, N, 3000, seed=5)
        want = oracle.linear_sampled(x, w, rows, cols) + b[cols]
        gu.assert_bitwise(got[rows, cols], want, f"bias gate_up M={M} sampled")


def test_bias_probes_on_gpu():
    from tests import oracle_pins as pins
    for p in pins.load_bias_probes():
        x, w = pins.probe_inputs(p)
        b = np.array([float.fromhex(p["b"])], dtype=np.float32)
        got = gu.bits(_run_bias(*gu.to_dev(x, w), _bias_dev(b)))[0, 0]
        assert got == int(p["expect_bits"], 16), (p["name"], hex(got))


def test_bias_null_and_alias_are_rejected():
    import torch
    import paper_2609_25624_amd as rg
    x, w = gu.layer(2, 64, 256, seed=1)
    xd, wd = gu.to_dev(x, w)
    y = torch.empty((2, 64), dtype=torch.float32, device=gu.dev())
    rc = rg.lib.rg_linear_bias(xd.data_ptr(), wd.data_ptr(), None, y.data_ptr(), 2, 64, 256,
                               torch.cuda.current_stream().cuda_stream)
    assert rc == rg.RG_ERR_INVAL
    rc = rg.lib.rg_linear_bias(xd.data_ptr(), wd.data_ptr(), y.data_ptr() + 4 * 64, y.data_ptr(), 2, 64, 256,
                               torch.cuda.current_stream().cuda_stream)
    assert rc == rg.RG_ERR_ALIAS
