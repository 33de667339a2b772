"""The CPU oracle against what the paper and the mathematics fix (no GPU)."""
import numpy as np
import pytest

import oracle
from tests import fp32_exact as fx
from tests import oracle_pins as pins


@pytest.mark.parametrize("name", sorted(pins.ALL_CHECKS))
def test_oracle_pin(name):
    fails = pins.ALL_CHECKS[name](oracle.lib())
    assert not fails, "\n".join(fails)


def test_probe_fixture_derivations_hold_in_exact_arithmetic():
    # The hand-derived expected bits also follow from the exact-rational emulation,
    # so a slip in a hand derivation cannot hide behind a matching oracle bug.
    for p in pins.load_probes():
        x, w = pins.probe_inputs(p)
        got = fx.float_bits(pins.emulated_dot(x[0], w[0]))
        assert got == int(p["expect_bits"], 16), p["name"]


def test_fp32_exact_helper_against_known_roundings():
    # IEEE-754 facts the emulator must reproduce (independent of any FPU).
    assert fx.float_bits(fx.add(2.0 ** 24, 1.0)) == 0x4B800000          # tie to even, down
    assert fx.float_bits(fx.add(2.0 ** 24 + 2, 1.0)) == 0x4B800002      # tie to even, up
    assert fx.float_bits(fx.fma(2.0 ** -100, 2.0 ** -49, 0.0)) == 0x00000001   # 2^-149, smallest subnormal
    assert fx.float_bits(fx.fma(2.0 ** -100, 2.0 ** -50, 0.0)) == 0x00000000   # 2^-150: tie, even is 0
    assert fx.float_bits(fx.fma(3.0 * 2.0 ** -100, 2.0 ** -50, 0.0)) == 0x00000002   # 3*2^-150: tie, up to even
    assert fx.float_bits(fx.fma(2.0 ** -100, 2.0 ** -49, 2.0 ** -149)) == 0x00000002
    assert fx.float_bits(fx.fma(-2.0 ** -100, 2.0 ** -60, 0.0)) == 0x80000000  # underflow keeps sign
    assert fx.float_bits(fx.add(-0.0, -0.0)) == 0x80000000
    assert fx.float_bits(fx.add(1.0, -1.0)) == 0x00000000
    assert fx.fma(2.0 ** 127, 4.0, 0.0) == float("inf")


def test_ref_fp64_matches_numpy_binary64():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((3, 517)).astype(np.float32)
    w = ((rng.standard_normal((4, 517)) * 0.02).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    y64, a = oracle.ref_fp64(x, w)
    wv = (w.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    prod = x.astype(np.float64)[:, None, :] * wv[None]
    assert np.allclose(y64, prod.sum(2), rtol=0, atol=1e-12 * np.abs(prod).sum(2).max())
    assert np.allclose(a, np.abs(prod).sum(2), rtol=1e-15)


def test_scaled_error_is_at_the_papers_ieee_level():
    # Supplement C, R1 table: IEEE-FMA error against FP64, scaled by the output
    # magnitude, is 4.8e-6; the accuracy section reports ~1e-7 relative error.
    # The documented order uses chains of at most 256 FMAs, so it sits at or below that.
    import synth
    x, w = synth.layer_inputs(4, 512, 4096, seed=0)
    y = oracle.linear(x, w)
    y64, _ = oracle.ref_fp64(x, w)
    scaled = np.abs(y - y64).max() / np.abs(y64).max()
    assert 1e-9 < scaled <= 4.8e-6
    rel = np.median(np.abs(y - y64) / np.abs(y64))
    assert rel < 1e-6


def test_k_up_to_one_segment_is_the_plain_sequential_fma_dot():
    # Special case: with K <= 256 there is one segment and no fold, i.e. the
    # textbook left-to-right fused dot product.
    rng = np.random.default_rng(9)
    for K in (1, 5, 64, 255, 256):
        x = rng.standard_normal(K).astype(np.float32)
        w = ((rng.standard_normal(K) * 0.02).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        acc = 0.0
        for k in range(K):
            acc = fx.fma(float(x[k]), fx.bf16_to_float(int(w[k])), acc)
        assert fx.float_bits(acc) == fx.float_bits(float(oracle.dot(x, w)))


def test_argmax_lowest_index_tie_break():
    assert oracle.argmax([1.0, 3.0, 3.0, 2.0]) == 1
    assert oracle.argmax([-1.0, -0.0, 0.0]) == 1          # -0 == +0: the lower index wins
    assert oracle.argmax([float("nan"), 2.0, 2.0]) == 1
    assert oracle.argmax([5.0]) == 0


def test_sampled_matches_full():
    import synth
    x, w = synth.layer_inputs(5, 300, 1000, seed=3)
    y = oracle.linear(x, w)
    rows = np.array([0, 4, 2, 3, 1])
    cols = np.array([0, 299, 150, 7, 100])
    s = oracle.linear_sampled(x, w, rows, cols)
    assert np.array_equal(s.view(np.uint32), y[rows, cols].view(np.uint32))
    with pytest.raises(IndexError):
        oracle.linear_sampled(x, w, [5], [0])


def test_gamma_values():
    # gamma_n, n = min(256,K) + ceil(K/256) - 1, u = 2^-24
    for K, want in [(1024, 1.54e-5), (4096, 1.62e-5), (8192, 1.71e-5), (14336, 1.85e-5), (28672, 2.19e-5)]:
        assert abs(oracle.gamma(K) - want) / want < 0.01
