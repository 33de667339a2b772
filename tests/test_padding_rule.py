"""The padding rule of the kernels, checked in exact rational arithmetic (no FPU).

Some kernels run a fixed number of steps and stage the steps past the data
with zeros: the register-tiled prefill kernel pads the short last 16-wide slab
of K, and the attention partials kernel pads a segment past the sequence's
last position.  Such a padded step must leave every chain value unchanged,
including -0, which a chain reaches when a negative product underflows (probe
O8: the first partial is taken as it is, so a -0 partial can reach y).

In binary32 round-to-nearest (IEEE 754, 6.3): fma(+0, -0, p) = -0 + p = p for
every p, but fma(+0, +0, -0) = +0.  So the padding must carry a -0 factor; the
tests below emulate the kernels' padded step sequences exactly and compare
them with the oracle.
"""
import numpy as np

import oracle
from tests import fp32_exact as fx


def _neg_zero_row(K):
    """x and W rows whose every 256-segment chain ends at -0 (probe O8 in every segment)."""
    x = np.full((1, K), -0.0, np.float32)
    w = np.full((1, K), 0x3F80, np.uint16)
    x[0, 0::256] = -(2.0 ** -100)
    w[0, 0::256] = 0x2180           # 2^-60: the product -2^-160 rounds to -0
    return x, w


def _chain_exact(xs, ws, start=0.0):
    p = start
    for a, b in zip(xs, ws):
        p = fx.fma(float(a), float(b), p)
    return p


def _tiled_steps(x, w, K, pad_w):
    """The prefill kernel's sequence: whole 16-wide slabs, k >= K staged as x = +0, w = pad_w."""
    KT = 16
    nsl = -(-K // KT)
    xs, ws = [], []
    for k in range(nsl * KT):
        if k < K:
            xs.append(float(x[0, k]))
            ws.append(fx.bf16_to_float(int(w[0, k])))
        else:
            xs.append(0.0)
            ws.append(pad_w)
    # segments of 256 (a slab never straddles one), folded left to right
    y = None
    for s in range(0, len(xs), 256):
        p = _chain_exact(xs[s:s + 256], ws[s:s + 256])
        y = p if y is None else fx.add(y, p)
    return y


def test_negative_zero_row_is_minus_zero_in_the_oracle():
    for K in (1, 8, 264, 1000, 4096):
        x, w = _neg_zero_row(K)
        assert int(oracle.linear(x, w).view(np.uint32)[0, 0]) == 0x80000000, K


def test_tiled_padding_with_minus_zero_weights_keeps_the_oracle_bits():
    for K in (8, 264, 1000):          # K % 16 == 8: the last slab is half padding
        x, w = _neg_zero_row(K)
        want = int(oracle.linear(x, w).view(np.uint32)[0, 0])
        got = fx.float_bits(_tiled_steps(x, w, K, pad_w=-0.0))
        assert got == want == 0x80000000, (K, hex(got))


def test_plus_zero_weight_padding_would_lose_the_sign():
    # the rule the kernel avoids: a +0 weight pad turns a -0 chain into +0
    for K in (8, 264, 1000):
        x, w = _neg_zero_row(K)
        assert fx.float_bits(_tiled_steps(x, w, K, pad_w=0.0)) == 0x00000000, K


def test_padded_step_identities():
    tiny = 2.0 ** -149
    for p in (0.0, -0.0, 1.0, -1.0, tiny, -tiny, 3.0e38):
        # weight pad -0 with x pad +0 (prefill kernel); e pad -0 with value pad +0 (attention)
        assert fx.float_bits(fx.fma(0.0, -0.0, p)) == fx.float_bits(p)
        assert fx.float_bits(fx.fma(-0.0, 0.0, p)) == fx.float_bits(p)
        # the segment sum of attention adds the pad e = -0 itself
        assert fx.float_bits(fx.add(p, -0.0)) == fx.float_bits(p)
    assert fx.float_bits(fx.fma(0.0, 0.0, -0.0)) == 0x00000000
    assert fx.float_bits(fx.add(-0.0, 0.0)) == 0x00000000


def test_attention_numerator_padding():
    """A segment numerator that is -0 (a tiny e times a tiny negative value underflows, then
    e * -0 terms) stays -0 through the padded positions only with a -0 pad on e."""
    e0 = float(np.float32(2.0 ** -29))
    v0 = fx.bf16_to_float(0x8001)    # -2^-133
    n = fx.fma(e0, v0, 0.0)          # -2^-162 rounds to -0
    assert fx.float_bits(n) == 0x80000000
    n = fx.fma(1.0, -0.0, n)
    assert fx.float_bits(n) == 0x80000000
    good, bad = n, n
    for _ in range(254):
        good = fx.fma(-0.0, 0.0, good)
        bad = fx.fma(0.0, 0.0, bad)
    assert fx.float_bits(good) == 0x80000000
    assert fx.float_bits(bad) == 0x00000000
