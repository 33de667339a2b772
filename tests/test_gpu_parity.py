"""GPU path (through the C-ABI) against the CPU oracle, bit for bit.

Configs follow the paper's probe and ablation shapes (Evaluation,
cross-architecture determinism; Supplement C): decode shapes of an
8B-parameter Llama-3-class model at M = 1, the same layers batched at
M = 4/16/64, an LM head with a near tie, 70B-class layers, and ragged shapes.
Inputs are seeded on the host and copied to the device (Supplement C, method).
"""
import numpy as np
import pytest

from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

L8B = {  # Llama-3-8B-shaped decode projections (N, K)
    "qkv": (6144, 4096),
    "o": (4096, 4096),
    "gate_up": (28672, 4096),
    "down": (4096, 14336),
}


@pytest.fixture(autouse=True)
def _reset_launch():
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(None)
    yield
    rg.rg_linear_set_launch(None)


def _check_layer(M, N, K, seed=0, w_std=0.02, layer_id=0, sampled=None):
    import torch
    gu.log(f"case M={M} N={N} K={K} seed={seed} layer={layer_id}")
    x, w = gu.layer(M, N, K, seed=seed, w_std=w_std, layer_id=layer_id)
    xd, wd = gu.to_dev(x, w)
    y = gu.run(xd, wd)
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    if sampled:
        import oracle
        rows, cols = gu.sample_indices(M, N, sampled, seed=seed)
        want = oracle.linear_sampled(x, w, rows, cols)
        gu.assert_bitwise(got[rows, cols], want, f"({M},{N},{K}) sampled")
    else:
        want = gu.oracle_full(x, w)
        gu.assert_bitwise(got, want, f"({M},{N},{K})")
    return x, w, got


def test_config1_small_layer():
    _check_layer(1, 1024, 1024)


@pytest.mark.parametrize("name", list(L8B))
def test_config2_8b_layers_m1(name):
    N, K = L8B[name]
    _check_layer(1, N, K, layer_id=list(L8B).index(name))


@pytest.mark.parametrize("M", [2, 3, 4, 16])
@pytest.mark.parametrize("name", list(L8B))
def test_config3_batched_rows_equal_single_row(name, M):
    # Row m of a batch is bitwise the single-row result (rule R4), and the batch matches the oracle.
    import torch
    N, K = L8B[name]
    x64, w = gu.layer(64, N, K, layer_id=list(L8B).index(name))
    x = x64[:M]                       # seeded rows: the M-row batch is a prefix of the 64-row one
    xd, wd = gu.to_dev(x, w)
    y = gu.run(xd, wd).cpu().numpy()
    want = gu.oracle_full(x, w)
    gu.assert_bitwise(y, want, f"{name} M={M}")
    for m in (0, M - 1):
        y1 = gu.run(xd[m:m + 1].contiguous(), wd)
        torch.cuda.synchronize()
        gu.assert_bitwise(y1.cpu().numpy()[0], y[m], f"{name} row {m} alone vs in batch {M}")


@pytest.mark.parametrize("name", list(L8B))
def test_config3_m64_full(name):
    """Every output of the M = 64 batch against the oracle's stored full-output digest, a sample
    against the definitional oracle computed here, and row 5 alone against row 5 in the batch."""
    import torch
    import oracle
    N, K = L8B[name]
    x, w = gu.layer(64, N, K, layer_id=list(L8B).index(name))
    xd, wd = gu.to_dev(x, w)
    y = gu.run(xd, wd)
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    gu.assert_full_output(got, x, w, f"{name}_m64")
    rows, cols = gu.sample_indices(64, N, 3000)
    gu.assert_bitwise(got[rows, cols], oracle.linear_sampled(x, w, rows, cols), f"{name} M=64 sampled")
    y1 = gu.run(xd[5:6].contiguous(), wd)
    gu.assert_bitwise(y1.cpu().numpy()[0], got[5], f"{name} row 5 at M=64 vs M=1")


@pytest.mark.parametrize("M", [4, 16])
@pytest.mark.parametrize("name", list(L8B))
def test_config3_full_output_digests(name, M):
    import torch
    N, K = L8B[name]
    x64, w = gu.layer(64, N, K, layer_id=list(L8B).index(name))
    x = np.ascontiguousarray(x64[:M])
    xd, wd = gu.to_dev(x, w)
    y = gu.run(xd, wd)
    torch.cuda.synchronize()
    gu.assert_full_output(y.cpu().numpy(), x, w, f"{name}_m{M}")


def test_config4_lm_head_m1_and_m16():
    import torch
    N, K = 128256, 4096
    x16, w = gu.layer(16, N, K, layer_id=7)
    xd, wd = gu.to_dev(x16, w)
    y16 = gu.run(xd, wd).cpu().numpy()
    y1 = gu.run(xd[:1].contiguous(), wd).cpu().numpy()
    torch.cuda.synchronize()
    want1 = gu.oracle_full(x16[:1], w)
    gu.assert_bitwise(y1, want1, "lm_head M=1")
    gu.assert_full_output(y1, x16[:1], w, "lm_head_m1")
    gu.assert_full_output(y16, x16, w, "lm_head_m16")
    import oracle
    rows, cols = gu.sample_indices(16, N, 4000)
    gu.assert_bitwise(y16[rows, cols], oracle.linear_sampled(x16, w, rows, cols), "lm_head M=16 sampled")
    gu.assert_bitwise(y16[0], y1[0], "lm_head row 0 at M=16 vs M=1")


def _near_tie_case(kstar, exact_tie, M):
    """W row n_b copies the argmax row n_a except one element k*, one bf16 ulp away.

    With exact_tie, x[:, k*] = 0 so both logits are bitwise equal and the lower index must win.
    """
    N, K = 128256, 4096
    x, w = gu.layer(M, N, K, layer_id=7)
    w = w.copy()
    x = x.copy()
    import oracle
    y0 = oracle.linear(x[:1], w)        # full row 0 of the unmodified logits
    na = oracle.argmax(y0[0])
    nb = N - 1 if na != N - 1 else 0
    lo, hi = min(na, nb), max(na, nb)
    w[hi] = w[lo]
    w[hi, kstar] = np.uint16((int(w[lo, kstar]) + 1) & 0xFFFF)   # one bf16 ulp (for finite, non-max values)
    if exact_tie:
        x[:, kstar] = 0.0
    return x, w, lo, hi


@pytest.mark.parametrize("kstar,exact_tie", [(0, False), (255, False), (256, False), (4095, False), (1000, True)])
def test_config4_near_tie_argmax(kstar, exact_tie):
    import torch
    import oracle
    import paper_2609_25624_amd as rg
    for M in (1, 16):
        x, w, lo, hi = _near_tie_case(kstar, exact_tie, M)
        xd, wd = gu.to_dev(x, w)
        y = gu.run(xd, wd)
        idx = torch.empty(M, dtype=torch.int64, device=xd.device)
        rg.rg_argmax_rows(y, idx)
        torch.cuda.synchronize()
        yh = y.cpu().numpy()
        rows = [0] if M == 1 else list(range(M))
        for m in rows:
            want = oracle.linear_sampled(x, w, [m, m], [lo, hi])
            gu.assert_bitwise(yh[m, [lo, hi]], want, f"near tie k*={kstar} row {m}")
        want_row0 = gu.oracle_full(x[:1], w)[0]
        gu.assert_bitwise(yh[0], want_row0, f"near tie k*={kstar} full row 0")
        assert int(idx[0].item()) == oracle.argmax(want_row0)
        if exact_tie:
            assert gu.bits(yh[0, lo]) == gu.bits(yh[0, hi])
            assert int(idx[0].item()) == lo or yh[0].max() > yh[0, lo]
        for m in rows:
            assert int(idx[m].item()) == oracle.argmax(yh[m])


@pytest.mark.parametrize("name,N,K", [("70b_gate_up", 57344, 8192), ("70b_down", 8192, 28672)])
def test_config5_70b_m1(name, N, K):
    x, w, got = _check_layer(1, N, K, w_std=0.01, layer_id=9)
    gu.assert_full_output(got, x, w, f"{name}_m1")


@pytest.mark.parametrize("name,N,K", [("70b_gate_up", 57344, 8192), ("70b_down", 8192, 28672)])
def test_config5_70b_m2048_full(name, N, K):
    """Every output of the 2048-row prefill layers against the oracle's stored full-output digest
    (on a mismatch the same-order vectorised oracle names the first differing output), and a
    sample against the definitional oracle computed here."""
    import torch
    import oracle
    import paper_2609_25624_amd as rg
    assert rg.rg_plan(2048, N, K)["kernel_name"] == "tiled"
    gu.log(f"case 70B {name} M=2048")
    x, w = gu.layer(2048, N, K, w_std=0.01, layer_id=9)
    xd, wd = gu.to_dev(x, w)
    y = gu.run(xd, wd)
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    del xd, wd, y
    gu.assert_full_output(got, x, w, f"{name}_m2048")
    rows, cols = gu.sample_indices(2048, N, 4000)
    gu.assert_bitwise(got[rows, cols], oracle.linear_sampled(x, w, rows, cols), f"{name} M=2048 sampled")


@pytest.mark.parametrize("M,N,K", [(65, 130, 1000), (100, 1000, 1000), (128, 256, 4096), (129, 257, 264),
                                   (300, 77, 520), (256, 4096, 4096), (2048, 192, 8200)])
def test_tiled_shapes(M, N, K):
    import paper_2609_25624_amd as rg
    assert rg.rg_plan(M, N, K)["kernel_name"] == "tiled"
    _check_layer(M, N, K, seed=M + K)


@pytest.mark.parametrize("M,N,K", [(2048, 4100, 264), (2000, 4096, 1032), (4096, 2048, 520)])
@pytest.mark.parametrize("depth,order", [(2, 0), (3, 0), (3, 1)])
def test_tiled_128_builds(M, N, K, depth, order):
    """The 128 x 128 prefill tile in both builds (two or three waves per SIMD), full outputs:
    ragged M and N tiles, a short last segment, a short last slab (K % 16 = 8, staged as +0),
    reversed workgroup order."""
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(kernel="tiled", depth=depth, grid_order=order)
    try:
        p = rg.rg_plan(M, N, K)
        assert (p["kernel_name"], p["tile_m"], p["depth"]) == ("tiled", 128, depth)
        _check_layer(M, N, K, seed=M + N + K + depth)
    finally:
        rg.rg_linear_set_launch(None)


@pytest.mark.parametrize("M", [1, 2, 3, 4, 5, 9])
@pytest.mark.parametrize("N,K", [(1, 8), (3, 16), (5, 248), (4, 256), (7, 264), (63, 1000), (65, 1016),
                                 (130, 4104), (33, 8200), (17, 520)])
def test_ragged_shapes(M, N, K):
    _check_layer(M, N, K, seed=M * 1000 + K)


@pytest.mark.parametrize("N", [1, 3, 4, 5, 1030, 2049])
@pytest.mark.parametrize("K", [4096, 4352, 5120, 8192, 12288])
def test_gemv_shapes(N, K):
    """M = 1 dense stream: ragged quads (N % 4), steps with fewer than 16 segments (K / 256 % 16),
    x in registers (K = 4096) or in LDS."""
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(kernel="gemv")
    try:
        assert rg.rg_plan(1, N, K)["kernel_name"] == "gemv"
        _check_layer(1, N, K, seed=N + K)
    finally:
        rg.rg_linear_set_launch(None)


@pytest.mark.parametrize("N,K,cfg", [
    (4120, 8192, dict()),                                   # 1030 quads on 129 x 4 waves: 2 or 1 each
    (4120, 12544, dict(waves_per_wg=4, grid_wgs=7)),        # 36-37 quads per wave, last step 1 segment
    (4096, 14336, dict()),                                  # one quad per wave, 3.5 steps
    (2049, 5120, dict(waves_per_wg=2, grid_wgs=300, grid_order=1)),   # empty workgroups
    (13, 8448, dict(waves_per_wg=1)),
])
def test_gemv_staged_x(N, K, cfg):
    """M = 1 dense stream with K > 4096: the workgroup's waves share each step's x part through
    LDS and walk the same steps; waves with fewer quads only move x in the rounds they sit out."""
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(kernel="gemv", **cfg)
    try:
        p = rg.rg_plan(1, N, K)
        gu.log(f"gemv staged x N={N} K={K} {cfg} -> waves {p['waves_per_wg']} grid {p['grid_wgs']}")
        _check_layer(1, N, K, seed=N ^ K)
    finally:
        rg.rg_linear_set_launch(None)


@pytest.mark.parametrize("M,kernel", [(1, "decode_xs"), (1, "decode"), (2, "decode")])
@pytest.mark.parametrize("N,K", [(1030, 4096), (4097, 1000), (515, 14336), (6141, 4352)])
@pytest.mark.parametrize("grid,order", [(3, 0), (7, 1), (13, 0)])
def test_round_major_quad_placement(M, kernel, N, K, grid, order):
    """The streaming decode kernels with four or more rounds per workgroup (quads placed
    round-major over the grid for one or two rows of x): even and uneven splits (Q % grid),
    a short last round, a last quad with fewer than 4 rows, reversed workgroup order."""
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(kernel=kernel, grid_wgs=grid, grid_order=order)
    try:
        p = rg.rg_plan(M, N, K)
        assert p["kernel_name"] == kernel
        Q = -(-N // 4)
        rounds = -(-(-(-Q // p["grid_wgs"])) // (p["rows_per_round"] // 4))
        assert rounds >= 4, rounds
        _check_layer(M, N, K, seed=M * 31 + N + K + grid)
    finally:
        rg.rg_linear_set_launch(None)


@pytest.mark.parametrize("M", [2, 5, 9, 16, 17, 33, 64, 100])
@pytest.mark.parametrize("N,K", [(3, 4096), (1030, 4104), (301, 8192), (130, 14336), (77, 520)])
@pytest.mark.parametrize("tile_n,waves,depth", [(0, 0, 0), (16, 4, 0), (16, 8, 0), (32, 0, 0), (64, 0, 0),
                                                (32, 0, 3), (64, 0, 3)])
def test_ktile_shapes(M, N, K, tile_n, waves, depth):
    """Small-M tiles with K shared out over thread groups: partial tiles in M and N, a short
    last segment (K % 256 != 0), rounds where only some groups have a segment (J % KS != 0),
    every tile width, 4 x 4 and 4 x 8 register tiles per thread (depth 3), and (forced) more
    than one tile of rows."""
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(kernel="ktile", tile_n=tile_n, waves_per_wg=waves, depth=depth)
    try:
        assert rg.rg_plan(M, N, K)["kernel_name"] == "ktile"
        _check_layer(M, N, K, seed=M * 7 + N + K)
    finally:
        rg.rg_linear_set_launch(None)


@pytest.mark.parametrize("M", [1, 2, 3, 4])
@pytest.mark.parametrize("N,K", [(1, 8), (9, 264), (1030, 4096), (33, 14336), (7, 4352), (515, 2056)])
def test_stream_kernel_bf16_shapes(M, N, K):
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(kernel="stream")
    try:
        assert rg.rg_plan(M, N, K)["kernel_name"] == "stream"
        _check_layer(M, N, K, seed=M * 7 + N + K)
    finally:
        rg.rg_linear_set_launch(None)


@pytest.mark.parametrize("K,kernel", [(4352, "gemv"), (4096, "gemv"), (4096, "decode_xs"), (4096, "stream")])
def test_order_probes_inside_m1_rows(K, kernel):
    """The hand-derived probes embedded in long rows (zero x and weight 1.0 around them) of an
    otherwise random 1030-row layer, run by the M = 1 streaming kernels and compared bitwise
    with the oracle on the same input."""
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(kernel=kernel)
    try:
        assert rg.rg_plan(1, 1030, K)["kernel_name"] == kernel
        _probes_in_rows(K, 1030)
    finally:
        rg.rg_linear_set_launch(None)


def _probes_in_rows(K, N):
    import torch
    import oracle
    from tests import oracle_pins as pins
    x0, w0 = gu.layer(1, N, K, seed=77)
    X = np.zeros((1, K), dtype=np.float32)
    W = np.array(w0, copy=True)
    for i, p in enumerate(pins.load_probes()):
        xp, wp = pins.probe_inputs(p)
        X[:] = 0.0
        X[0, :xp.shape[1]] = xp[0]
        row = 3 + 97 * i
        W[row] = 0x3F80
        W[row, :wp.shape[1]] = wp[0]
        xd, wd = gu.to_dev(X, W)
        y = gu.run(xd, wd)
        torch.cuda.synchronize()
        want = oracle.linear_sampled(X, W, np.array([0]), np.array([row]))
        got = gu.bits(y.cpu().numpy())[0, row]
        assert int(got) == int(gu.bits(want)[0]), f"{p['name']} row {row}"


@pytest.mark.parametrize("M,N,K", [(1, 10, 7), (2, 33, 301), (3, 5, 1), (1, 4, 257), (100, 1000, 1000)])
def test_generic_shapes(M, N, K):
    _check_layer(M, N, K, seed=K)


def test_misaligned_pointers_take_the_generic_path():
    import torch
    M, N, K = 2, 37, 1024
    x, w = gu.layer(M, N, K, seed=11)
    xb = torch.zeros(M * K + 1, dtype=torch.float32, device=gu.dev())
    xb[1:] = torch.from_numpy(np.array(x, copy=True).ravel()).to(gu.dev())
    xd = xb[1:].view(M, K)                      # 4-byte but not 16-byte aligned
    wd = gu.to_dev(x, w)[1]
    y = gu.run(xd, wd)
    gu.assert_bitwise(y.cpu().numpy(), gu.oracle_full(x, w), "misaligned x")


def test_order_probes_on_gpu():
    # The hand-derived probes (tests/golden) also hold on the GPU, alone and placed
    # at row m=5 of a 16-row batch and row n=1000 of a 4096-row W (position independence).
    import torch
    from tests import oracle_pins as pins
    for p in pins.load_probes():
        x1, w1 = pins.probe_inputs(p)
        want = int(p["expect_bits"], 16)
        xd, wd = gu.to_dev(x1, w1)
        got = int(gu.bits(gu.run(xd, wd).cpu().numpy())[0, 0])
        assert got == want, f"{p['name']} alone: 0x{got:08x}"
        K = x1.shape[1]
        X, W = gu.layer(16, 4096, K, seed=5)
        X = X.copy(); W = W.copy()
        X[5] = x1[0]
        W[1000] = w1[0]
        xd, wd = gu.to_dev(X, W)
        y = gu.run(xd, wd)
        torch.cuda.synchronize()
        got = int(gu.bits(y.cpu().numpy())[5, 1000])
        assert got == want, f"{p['name']} placed: 0x{got:08x}"


def _launch_settings():
    return [
        dict(),
        dict(waves_per_wg=1, depth=2),
        dict(waves_per_wg=2, grid_wgs=97),
        dict(waves_per_wg=4, grid_wgs=600, depth=2, grid_order=1),
        dict(grid_wgs=1),
        dict(kernel="decode"),
        dict(kernel="decode", waves_per_wg=7, grid_wgs=300),
        dict(kernel="decode_xs", waves_per_wg=6),
        dict(kernel="decode_xs", waves_per_wg=2, depth=3, grid_wgs=1000, grid_order=1),
        dict(kernel="tiled"),
        dict(kernel="tiled", grid_order=1),
        dict(kernel="generic"),
        dict(kernel="generic", grid_wgs=3, grid_order=1),
        dict(kernel="gemv"),
        dict(kernel="gemv", waves_per_wg=1, grid_wgs=5, grid_order=1),
        dict(kernel="gemv", waves_per_wg=2, grid_wgs=1000),
        dict(kernel="gemv", waves_per_wg=3, grid_wgs=256, grid_order=1),
        dict(kernel="ktile"),
        dict(kernel="ktile", tile_n=16, grid_order=1),
        dict(kernel="ktile", tile_n=32),
        dict(kernel="ktile", tile_n=64, grid_order=1),
        dict(kernel="ktile", tile_n=16, waves_per_wg=8),
        dict(kernel="ktile", tile_n=32, depth=3),
        dict(kernel="ktile", tile_n=64, depth=3, grid_order=1),
        dict(kernel="stream"),
        dict(kernel="stream", grid_wgs=7, grid_order=1),
        dict(kernel="skinny"),
        dict(kernel="skinny", depth=3, grid_order=1),
        dict(kernel="skinny", depth=2, grid_wgs=5),
        dict(kernel="skinny", waves_per_wg=8, grid_wgs=1000, grid_order=1),
        dict(kernel="skinny", slice_m=1),
        dict(kernel="wtile"),
        dict(kernel="wtile", grid_order=1),
        dict(kernel="wtile", waves_per_wg=8),
    ]


@pytest.mark.parametrize("M,N,K", [(1, 6144, 4096), (1, 1029, 4096), (1, 4096, 14336), (1, 1030, 4352), (3, 1000, 1000), (4, 2048, 2560),
                                   (16, 2048, 4096), (37, 1030, 4352), (70, 1024, 1024)])
def test_launch_settings_do_not_change_bits(M, N, K):
    import torch
    import paper_2609_25624_amd as rg
    x, w = gu.layer(M, N, K, seed=21)
    xd, wd = gu.to_dev(x, w)
    want = gu.oracle_full(x, w)
    for cfg in _launch_settings():
        rg.rg_linear_set_launch(**cfg) if cfg else rg.rg_linear_set_launch(None)
        try:
            plan = rg.rg_plan(M, N, K)
        except rg.RgError:
            continue                                # setting not valid for this shape
        gu.log(f"  launch {cfg} -> {plan['kernel_name']} nw={plan['waves_per_wg']} grid={plan['grid_wgs']}")
        y = gu.run(xd, wd)
        torch.cuda.synchronize()
        gu.assert_bitwise(y.cpu().numpy(), want, f"({M},{N},{K}) launch {cfg}")
    rg.rg_linear_set_launch(None)


def test_cu_masks_do_not_change_bits():
    import torch
    import paper_2609_25624_amd as rg
    ncu = rg.rg_device_cu_count()
    nwords = (ncu + 31) // 32
    masks = {
        "all": [0xFFFFFFFF] * nwords,
        "half": [0xFFFFFFFF if i < nwords // 2 else 0 for i in range(nwords)],
        "37": [(1 << 32) - 1 if i == 0 else ((1 << 5) - 1 if i == 1 else 0) for i in range(nwords)],
        "alternate": [0x55555555] * nwords,
        "first64": [0xFFFFFFFF if i < 2 else 0 for i in range(nwords)],
    }
    # the M = 1 step's QKV layer, two slices of the skinny kernel, and the wave-tile kernel
    cases = [((1, 6144, 4096), None), ((16, 2048, 4096), None), ((40, 1030, 4096), dict(kernel="wtile"))]
    done = 0
    for (M, N, K), cfg in cases:
        rg.rg_linear_set_launch(**cfg) if cfg else rg.rg_linear_set_launch(None)
        x, w = gu.layer(M, N, K, seed=31)
        xd, wd = gu.to_dev(x, w)
        want = gu.oracle_full(x, w)
        for name, mask in masks.items():
            try:
                s = rg.rg_stream_create_cu_mask(mask)
            except rg.RgError as e:
                gu.log(f"  cu mask {name}: the runtime refused it ({e})")
                continue
            try:
                ext = torch.cuda.ExternalStream(s)
                y = torch.empty((M, N), dtype=torch.float32, device=gu.dev())
                torch.cuda.synchronize()
                gu.run(xd, wd, stream=ext, out=y)
                ext.synchronize()
                gu.log(f"  ({M},{N},{K}) {rg.rg_plan(M, N, K)['kernel_name']} cu mask {name}: done")
                gu.assert_bitwise(y.cpu().numpy(), want, f"({M},{N},{K}) cu mask {name}")
                done += 1
            finally:
                torch.cuda.synchronize()
                rg.rg_stream_destroy(s)
    rg.rg_linear_set_launch(None)
    assert done >= 9, "fewer than three CU masks per case could be exercised"


def test_fifty_repeats_one_distinct_output():
    # Supplement C, R3 ablation: ordered split-K returns one result in 50 runs.
    import torch
    M, N, K = 1, 4096, 14336
    x, w = gu.layer(M, N, K, seed=41)
    xd, wd = gu.to_dev(x, w)
    outs = torch.empty((50, N), dtype=torch.float32, device=gu.dev())
    for r in range(50):
        gu.run(xd, wd, out=outs[r:r + 1])
    torch.cuda.synchronize()
    o = outs.cpu().numpy()
    assert len({o[r].tobytes() for r in range(50)}) == 1
    gu.assert_bitwise(o[0:1], gu.oracle_full(x, w), "repeat")


def test_alternating_inputs_never_see_stale_data():
    import torch
    M, N, K = 1, 4096, 4096
    xa, wa = gu.layer(M, N, K, seed=51)
    xb, wb = gu.layer(M, N, K, seed=52)
    da, db = gu.to_dev(xa, wa), gu.to_dev(xb, wb)
    ya_want, yb_want = gu.oracle_full(xa, wa), gu.oracle_full(xb, wb)
    outs = []
    for r in range(10):
        d = da if r % 2 == 0 else db
        outs.append(gu.run(*d))
    torch.cuda.synchronize()
    for r, y in enumerate(outs):
        gu.assert_bitwise(y.cpu().numpy(), ya_want if r % 2 == 0 else yb_want, f"alternating call {r}")


def test_other_stream_and_concurrent_load():
    import torch
    M, N, K = 2, 28672, 4096
    x, w = gu.layer(M, N, K, seed=61)
    xd, wd = gu.to_dev(x, w)
    want = gu.oracle_full(x, w)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    a = torch.randn(4096, 4096, device=gu.dev())
    torch.cuda.synchronize()
    ys = []
    with torch.cuda.stream(s2):
        for _ in range(8):
            a = a @ a.t()
            a = a / a.abs().max()
    with torch.cuda.stream(s1):
        for _ in range(4):
            ys.append(gu.run(xd, wd, stream=s1))
    torch.cuda.synchronize()
    for y in ys:
        gu.assert_bitwise(y.cpu().numpy(), want, "stream under load")


def test_cast_kernel_is_the_exact_upcast():
    import torch
    import paper_2609_25624_amd as rg
    rng = np.random.default_rng(3)
    w = rng.integers(0, 1 << 16, 100003, dtype=np.uint32).astype(np.uint16)
    wd = torch.from_numpy(w.view(np.int16)).to(gu.dev())
    out = torch.empty(w.size, dtype=torch.float32, device=gu.dev())
    rg.rg_cast_bf16_f32(wd, out)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy().view(np.uint32), w.astype(np.uint32) << 16)


def test_argmax_kernel_ties_and_nan():
    import torch
    import oracle
    import paper_2609_25624_amd as rg
    rows = [
        [1.0, 3.0, 3.0, 2.0],
        [-1.0, -0.0, 0.0, -5.0],
        [float("nan"), 2.0, 2.0, 1.0],
        [float("nan")] * 4,
    ]
    y = torch.tensor(rows, dtype=torch.float32, device=gu.dev())
    idx = torch.empty(4, dtype=torch.int64, device=gu.dev())
    rg.rg_argmax_rows(y, idx)
    torch.cuda.synchronize()
    assert idx.cpu().tolist() == [1, 1, 1, -1]
    big = np.full((3, 100000), -1.0, dtype=np.float32)
    big[0, 99999] = 2.0
    big[1, [17, 50000, 99999]] = 5.0
    big[2, :] = 0.0
    yb = torch.from_numpy(big).to(gu.dev())
    idx = torch.empty(3, dtype=torch.int64, device=gu.dev())
    rg.rg_argmax_rows(yb, idx)
    torch.cuda.synchronize()
    assert idx.cpu().tolist() == [oracle.argmax(big[i]) for i in range(3)] == [99999, 17, 0]


@pytest.mark.parametrize("N,offset", [(128256, 0), (100003, 0), (128256, 1), (7, 0), (65540, 0)])
def test_argmax_kernel_paths(N, offset):
    # 16-byte loads where the row length is a multiple of 4 and the rows are 16-byte aligned,
    # 4-byte loads otherwise (offset 1 shifts the rows off alignment); ties and NaNs in every
    # position of a 16-byte vector, and the winner in the last element
    import torch
    import oracle
    import paper_2609_25624_amd as rg
    rng = np.random.default_rng(N + offset)
    M = 6
    y = rng.standard_normal((M, N)).astype(np.float32)
    y[0, :] = 1.0                                   # all tied: index 0
    y[1, [N - 1, N // 2]] = 9.0                     # tie: the lower index
    y[2, ::3] = np.nan                              # NaNs never win
    y[3, N - 1] = 50.0                              # the winner is the last element
    y[4, :] = np.nan
    y[4, min(N - 1, 5)] = -3.0                      # one number among NaNs
    flat = np.zeros(M * N + offset, dtype=np.float32)
    flat[offset:] = y.ravel()
    base = torch.from_numpy(flat).to(gu.dev())
    yd = base[offset:].view(M, N)
    idx = torch.empty(M, dtype=torch.int64, device=gu.dev())
    rg.rg_argmax_rows(yd, idx)
    torch.cuda.synchronize()
    assert idx.cpu().tolist() == [oracle.argmax(y[i]) for i in range(M)]
