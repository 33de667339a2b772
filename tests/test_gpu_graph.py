"""The library's calls captured in a HIP graph (torch.cuda.CUDAGraph) and replayed.

rg_linear and rg_attn_decode allocate nothing and never synchronize, so they can be
recorded in a graph.  The graph is replayed several times with eager calls and
synchronizations between the replays, and every replay must give the eager results
bit for bit (which equal the oracle).
"""
import numpy as np
import pytest

import synth
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

_SHAPES = [(1, 1030, 4096), (1, 777, 14336), (4, 512, 1000), (16, 515, 4104), (70, 130, 1000)]


def test_linear_and_attention_in_a_replayed_graph():
    import torch
    import oracle
    import paper_2609_25624_amd as rg
    gu.log("graph: capture rg_linear x5 + rg_attn_decode, replay 3 times")
    layers = []
    for i, (M, N, K) in enumerate(_SHAPES):
        x, w = gu.layer(M, N, K, seed=60 + i)
        xd, wd = gu.to_dev(x, w)
        layers.append((xd, wd, gu.oracle_full(x, w), M, N))
    B, H, Hkv, Lmax, D = 3, 8, 2, 600, 128
    lens = np.array([600, 257, 1], np.int32)
    q, kc, vc = synth.attn_inputs(B, H, Hkv, Lmax, D, seed=61)
    scale = np.float32(1.0 / np.sqrt(D))
    want_attn = oracle.attn_decode(q, kc, vc, lens, scale)
    qd = torch.from_numpy(q.copy()).to(gu.dev())
    kd = torch.from_numpy(kc.view(np.int16).copy()).to(gu.dev())
    vd = torch.from_numpy(vc.view(np.int16).copy()).to(gu.dev())
    ld = torch.from_numpy(lens.copy()).to(gu.dev())
    ws = torch.empty(rg.rg_attn_workspace_size(B, H, Lmax, D), dtype=torch.uint8, device=gu.dev())

    ys = [torch.empty((M, N), dtype=torch.float32, device=gu.dev()) for (_, _, _, M, N) in layers]
    ao = torch.empty((B, H, D), dtype=torch.float32, device=gu.dev())

    def step():
        for (xd, wd, _, _, _), y in zip(layers, ys):
            rg.rg_linear(xd, wd, y)
        rg.rg_attn_decode(qd, kd, vd, ld, ao, scale, workspace=ws)

    # eager results first (these equal the oracle)
    step()
    torch.cuda.synchronize()
    eager = [y.cpu().numpy().copy() for y in ys]
    eager_attn = ao.cpu().numpy().copy()
    for (_, _, want, _, _), got, shape in zip(layers, eager, _SHAPES):
        gu.assert_bitwise(got, want, f"eager {shape}")
    assert np.array_equal(gu.bits(eager_attn), gu.bits(want_attn)), "eager attention"

    # capture on a side stream (torch's graph capture), after a warm-up call on that stream
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    for r in range(3):
        for y in ys:
            y.fill_(float("nan"))                 # the replay must overwrite every output
        ao.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for y, want, shape in zip(ys, eager, _SHAPES):
            assert np.array_equal(gu.bits(y.cpu().numpy()), gu.bits(want)), f"replay {r} {shape}"
        assert np.array_equal(gu.bits(ao.cpu().numpy()), gu.bits(eager_attn)), f"replay {r} attention"
        # eager work between replays, as a program would do
        xd, wd, want, M, N = layers[0]
        z = torch.empty((M, N), dtype=torch.float32, device=gu.dev())
        rg.rg_linear(xd, wd, z)
        torch.cuda.synchronize()
        gu.assert_bitwise(z.cpu().numpy(), want, f"eager call after replay {r}")
