"""The same-order vectorised oracle (oracle/rg_oracle_fast.c) is bit-identical to the definitional
oracle (oracle/rg_oracle.c) on every shape class: ragged K around the 256-segment boundaries, N not
a multiple of its 16-output blocks, M not a multiple of its 4- and 128-row blocks, the hand-derived
order probes, signed zeros through underflow, subnormal inputs and results, integer-exact inputs,
large magnitudes, and thread counts.  That pin is what lets the GPU tests compare the largest
workloads output for output."""
import numpy as np
import pytest

import oracle
import synth
from tests import oracle_pins as pins

pytestmark = pytest.mark.skipif(not oracle.fast_supported(), reason="host CPU lacks AVX2/FMA")


def _same(a, b, what):
    ba, bb = a.view(np.uint32), b.view(np.uint32)
    bad = np.flatnonzero(ba.ravel() != bb.ravel())
    assert bad.size == 0, f"{what}: {bad.size} differ, first flat {bad[0]}: 0x{ba.ravel()[bad[0]]:08x} vs 0x{bb.ravel()[bad[0]]:08x}"


@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (1, 17, 255), (3, 16, 256), (5, 33, 257), (4, 15, 511),
                                   (129, 31, 300), (7, 100, 1000), (2, 1030, 4096), (9, 3, 4104),
                                   (130, 65, 520), (1, 5, 14336)])
def test_random_shapes(M, N, K):
    x, w = synth.layer_inputs(M, N, K, seed=M * 7 + N + K)
    _same(oracle.linear_fast(x, w), oracle.linear(x, w), f"({M},{N},{K})")


def test_threads_do_not_change_bits():
    x, w = synth.layer_inputs(37, 70, 777, seed=3)
    want = oracle.linear(x, w)
    for t in (1, 2, 3, 8):
        _same(oracle.linear_fast(x, w, nthreads=t), want, f"{t} threads")


def test_order_probes():
    for p in pins.load_probes():
        x, w = pins.probe_inputs(p)
        got = int(oracle.linear_fast(x, w).view(np.uint32)[0, 0])
        assert got == int(p["expect_bits"], 16), p["name"]


def test_probes_in_every_lane_and_row_block():
    # each probe placed at every lane of a 16-output block and in rows of both 4-row halves
    for p in pins.load_probes():
        x1, w1 = pins.probe_inputs(p)
        K = x1.shape[1]
        x, w = synth.layer_inputs(9, 35, K, seed=11)
        x, w = x.copy(), w.copy()
        x[5] = x1[0]
        for n in range(0, 35, 3):
            w[n] = w1[0]
        _same(oracle.linear_fast(x, w), oracle.linear(x, w), p["name"])


def test_signed_zero_subnormal_and_large_values():
    rng = np.random.default_rng(5)
    M, N, K = 6, 40, 600
    x = rng.choice(np.array([-0.0, 0.0, 2.0 ** -100, -(2.0 ** -100), 2.0 ** -149, 1e30, -1e30, 1.0],
                            dtype=np.float32), size=(M, K))
    w = rng.choice(np.array([0x8000, 0x0000, 0x2180, 0xA180, 0x0001, 0x8001, 0x3F80, 0x7F00],
                            dtype=np.uint16), size=(N, K))
    x[0] = -0.0
    x[0, 0::256] = -(2.0 ** -100)
    w[0] = 0x3F80
    w[0, 0::256] = 0x2180                      # every segment of (0, 0) ends at -0
    want = oracle.linear(x, w)
    assert int(want.view(np.uint32)[0, 0]) == 0x80000000
    _same(oracle.linear_fast(x, w), want, "special values")


def test_integer_exact_inputs():
    M, N, K = 5, 21, 1300
    m = np.arange(M)[:, None]
    n = np.arange(N)[:, None]
    k = np.arange(K)[None, :]
    x = (((3 * m + k) % 7) - 3).astype(np.float32)
    wf = (((n + 2 * k) % 5) - 2).astype(np.float32)
    w = (wf.view(np.uint32) >> 16).astype(np.uint16)
    y = oracle.linear_fast(x, w)
    assert np.array_equal(y, (x.astype(np.float64) @ wf.astype(np.float64).T).astype(np.float32))
    _same(y, oracle.linear(x, w), "integers")
