"""Pins that tie the CPU oracle to things other than itself.

Every check takes a loaded oracle library (ctypes CDLL exposing rg_oracle_dot
and rg_oracle_linear), so the same checks run against the real oracle and
against deliberately broken copies of it (tests/test_oracle_mutants.py).
Each check returns a list of failure strings (empty = pass).

What pins what:
  * hand-derived probes (tests/golden/order_probes.json): the segment length,
    the in-segment sequential order, the left fold, the +0 start, subnormals;
  * binary64 reference within gamma_n * sum|x*w| (Higham's inner-product
    bound): no dropped, doubled or misplaced term, on many ragged K;
  * integer-valued inputs: every order gives the exact integer, so a wrong
    operand pairing, transposition or index shows up as a wrong integer;
  * exact-rational emulation of binary32 FMA and addition on tiny inputs:
    correct rounding, signed zeros and gradual underflow of the C library;
  * invariants: rows of x and of W permute outputs; a batch is its rows;
  * the bias variant: hand-derived probes (tests/golden/bias_probes.json),
    exact integers, and b = 0;
  * FP32 weights: hand-derived probes (tests/golden/f32w_probes.json), the
    order probes with widened weights, exact emulation, the binary64 bound,
    integers beyond bfloat16 precision, and agreement with the BF16 path on
    widened BF16 weights.
"""
import ctypes
import json
import os
import struct

import numpy as np

from tests import fp32_exact as fx

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "order_probes.json")
CHUNK = 256
U32 = 2.0 ** -24


def _setup(L):
    vp, i64, ci = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    L.rg_oracle_dot.argtypes = [vp, vp, i64]
    L.rg_oracle_dot.restype = ctypes.c_float
    L.rg_oracle_linear.argtypes = [vp, vp, vp, i64, i64, i64, ci]
    L.rg_oracle_linear.restype = ci
    return L


def _linear(L, x, w, nthreads=4):
    x = np.ascontiguousarray(x, dtype=np.float32)
    w = np.ascontiguousarray(w, dtype=np.uint16)
    M, K = x.shape
    N = w.shape[0]
    y = np.empty((M, N), dtype=np.float32)
    rc = L.rg_oracle_linear(x.ctypes.data, w.ctypes.data, y.ctypes.data, M, N, K, nthreads)
    assert rc == 0
    return y


def f32_bits(v) -> int:
    return struct.unpack("<I", struct.pack("<f", float(v)))[0]


def load_probes():
    with open(GOLDEN) as f:
        return json.load(f)["probes"]


def probe_inputs(p):
    K = p["K"]
    x = np.zeros((1, K), dtype=np.float32)
    w = np.full((1, K), 0x3F80, dtype=np.uint16)
    for a, b, v in p["x"]:
        x[0, a:b] = float.fromhex(v)
    for a, b, v in p.get("w", []):
        w[0, a:b] = int(v, 16)
    return x, w


def check_probes(L):
    L = _setup(L)
    fails = []
    for p in load_probes():
        x, w = probe_inputs(p)
        got = f32_bits(_linear(L, x, w)[0, 0])
        want = int(p["expect_bits"], 16)
        if got != want:
            fails.append(f"{p['name']}: got 0x{got:08x} want 0x{want:08x}")
    return fails


def gamma(K):
    J = -(-K // CHUNK)
    n = min(CHUNK, K) + J - 1
    return n * U32 / (1.0 - n * U32)


def check_fp64_bound(L, Ks=None, seed=0):
    """|y - y64| <= gamma_n * sum|x w| (+ the binary64 sum's own error) on ragged K."""
    L = _setup(L)
    rng = np.random.default_rng(seed)
    if Ks is None:
        Ks = [1, 2, 7, 8, 9, 100, 255, 256, 257, 300, 511, 512, 513, 600, 1000, 1024, 1500, 2048, 4100]
    fails = []
    for K in Ks:
        M, N = 3, 5
        x = rng.standard_normal((M, K)).astype(np.float32)
        wf = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
        w = (wf.view(np.uint32) >> 16).astype(np.uint16)    # truncation is fine for inputs
        y = _linear(L, x, w).astype(np.float64)
        wv = (w.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        prod = x.astype(np.float64)[:, None, :] * wv[None, :, :]           # exact in binary64
        y64 = prod.sum(axis=2)
        a = np.abs(prod).sum(axis=2)
        g64 = K * 2.0 ** -53 / (1 - K * 2.0 ** -53)
        bound = gamma(K) * a + g64 * a
        err = np.abs(y - y64)
        if not np.all(err <= bound):
            i = np.unravel_index(np.argmax(err - bound), err.shape)
            fails.append(f"K={K}: |y-y64|={err[i]:.3e} > bound {bound[i]:.3e}")
    return fails


def check_integer_exact(L):
    """Small integers: all partial sums are exact, so y is the integer dot product in any order."""
    L = _setup(L)
    fails = []
    for (M, N, K) in [(3, 4, 5), (2, 7, 256), (4, 3, 257), (5, 6, 700), (1, 9, 1000)]:
        m = np.arange(M)[:, None]
        n = np.arange(N)[:, None]
        k = np.arange(K)[None, :]
        xi = ((3 * m + k) % 7) - 3
        wi = ((n + 2 * k) % 5) - 2
        x = xi.astype(np.float32)
        w = (wi.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)   # exact in bf16
        want = xi.astype(np.int64) @ wi.astype(np.int64).T
        got = _linear(L, x, w)
        if not np.array_equal(got.astype(np.int64), want) or not np.all(got == want):
            fails.append(f"integer-exact ({M},{N},{K}) mismatch")
    return fails


def emulated_dot(xr, wr):
    """The documented order on exact rationals: segment chains of fma, then a left fold."""
    K = len(xr)
    y = None
    for k0 in range(0, K, CHUNK):
        p = 0.0
        for k in range(k0, min(k0 + CHUNK, K)):
            p = fx.fma(float(xr[k]), fx.bf16_to_float(int(wr[k])), p)
        y = p if y is None else fx.add(y, p)
    return y


def check_exact_emulation(L, seed=1):
    """Tiny random and adversarial rows: oracle bits == exact-rational emulation bits."""
    L = _setup(L)
    rng = np.random.default_rng(seed)
    fails = []
    cases = []
    for K in (1, 3, 17, 256, 257, 520):
        x = rng.standard_normal(K).astype(np.float32)
        w = ((rng.standard_normal(K) * 0.02).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        cases.append((f"normal K={K}", x, w))
    # wide dynamic range with subnormal products and cancellations
    K = 300
    x = (rng.standard_normal(K) * 2.0 ** rng.integers(-70, 40, K)).astype(np.float32)
    w = ((rng.standard_normal(K) * 2.0 ** rng.integers(-80, 10, K)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    cases.append(("wide range", x, w))
    x = np.array([1e-30, -1e-30, 3.0, -3.0] * 80, dtype=np.float32)
    w = np.array([0x0001, 0x8001, 0x3F80, 0x3F80] * 80, dtype=np.uint16)
    cases.append(("subnormal weights, cancellation", x, w))
    for name, x, w in cases:
        got = f32_bits(L.rg_oracle_dot(np.ascontiguousarray(x).ctypes.data, np.ascontiguousarray(w).ctypes.data, len(x)))
        want = f32_bits(emulated_dot(x, w))
        if got != want:
            fails.append(f"{name}: got 0x{got:08x} want 0x{want:08x}")
    return fails


def check_invariants(L, seed=2):
    """Row permutations of x and W permute y; a batch equals its rows computed alone."""
    L = _setup(L)
    rng = np.random.default_rng(seed)
    M, N, K = 6, 7, 777
    x = rng.standard_normal((M, K)).astype(np.float32)
    w = ((rng.standard_normal((N, K)) * 0.02).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    y = _linear(L, x, w)
    fails = []
    pm, pn = rng.permutation(M), rng.permutation(N)
    yp = _linear(L, x[pm], w[pn])
    if not np.array_equal(yp.view(np.uint32), y[pm][:, pn].view(np.uint32)):
        fails.append("row permutation changed bits")
    for m in range(M):
        y1 = _linear(L, x[m:m + 1], w)
        if not np.array_equal(y1.view(np.uint32), y[m:m + 1].view(np.uint32)):
            fails.append(f"row {m} alone differs from the batch")
    return fails


BIAS_GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "bias_probes.json")


def _linear_bias(L, x, w, b, nthreads=4):
    vp, i64, ci = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    L.rg_oracle_linear_bias.argtypes = [vp, vp, vp, vp, i64, i64, i64, ci]
    L.rg_oracle_linear_bias.restype = ci
    x = np.ascontiguousarray(x, dtype=np.float32)
    w = np.ascontiguousarray(w, dtype=np.uint16)
    b = np.ascontiguousarray(b, dtype=np.float32)
    M, K = x.shape
    N = w.shape[0]
    y = np.empty((M, N), dtype=np.float32)
    assert L.rg_oracle_linear_bias(x.ctypes.data, w.ctypes.data, b.ctypes.data, y.ctypes.data, M, N, K, nthreads) == 0
    return y


def load_bias_probes():
    with open(BIAS_GOLDEN) as f:
        return json.load(f)["probes"]


def check_bias(L, seed=5):
    """The bias variant: the hand-derived probes (tests/golden/bias_probes.json), exact
    integers (every order of the sum gives the same integer, so only the additions
    themselves are tested), and the bias-free product where b = 0 (x + 0 == x)."""
    L = _setup(L)
    fails = []
    for p in load_bias_probes():
        x, w = probe_inputs(p)
        b = np.array([float.fromhex(p["b"])], dtype=np.float32)
        got = f32_bits(_linear_bias(L, x, w, b)[0, 0])
        want = int(p["expect_bits"], 16)
        if got != want:
            fails.append(f"{p['name']}: got 0x{got:08x} want 0x{want:08x}")
    rng = np.random.default_rng(seed)
    M, N, K = 3, 9, 600
    xi = rng.integers(-8, 9, (M, K)).astype(np.float32)
    wi = rng.integers(-4, 5, (N, K)).astype(np.float32)
    bi = rng.integers(-1000, 1001, N).astype(np.float32)
    w16 = (wi.view(np.uint32) >> 16).astype(np.uint16)
    got = _linear_bias(L, xi, w16, bi)
    want = (xi.astype(np.int64) @ wi.astype(np.int64).T + bi.astype(np.int64)).astype(np.float32)
    if not np.array_equal(got, want):
        fails.append("integer-valued inputs with an integer bias are not exact")
    x = rng.standard_normal((M, K)).astype(np.float32)
    w = ((rng.standard_normal((N, K)) * 0.02).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    y0 = _linear_bias(L, x, w, np.zeros(N, dtype=np.float32))
    y = _linear(L, x, w)
    if not np.array_equal(y0.view(np.uint32), (y + np.float32(0.0)).view(np.uint32)):
        fails.append("b = 0 changed a nonzero output")
    return fails


F32W_GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "f32w_probes.json")


def _linear_f32w(L, x, w, nthreads=4):
    vp, i64, ci = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    L.rg_oracle_linear_f32w.argtypes = [vp, vp, vp, i64, i64, i64, ci]
    L.rg_oracle_linear_f32w.restype = ci
    x = np.ascontiguousarray(x, dtype=np.float32)
    w = np.ascontiguousarray(w, dtype=np.float32)
    M, K = x.shape
    N = w.shape[0]
    y = np.empty((M, N), dtype=np.float32)
    assert L.rg_oracle_linear_f32w(x.ctypes.data, w.ctypes.data, y.ctypes.data, M, N, K, nthreads) == 0
    return y


def load_f32w_probes():
    with open(F32W_GOLDEN) as f:
        return json.load(f)["probes"]


def f32w_probe_inputs(p):
    K = p["K"]
    x = np.zeros((1, K), dtype=np.float32)
    w = np.ones((1, K), dtype=np.float32)
    for a, b, v in p["x"]:
        x[0, a:b] = float.fromhex(v)
    wb = w.view(np.uint32)
    for a, b, v in p.get("w", []):
        wb[0, a:b] = int(v, 16)
    return x, w


def emulated_dot_f32w(xr, wr):
    """The documented order on exact rationals with float32 weights used as they are."""
    K = len(xr)
    y = None
    for k0 in range(0, K, CHUNK):
        p = 0.0
        for k in range(k0, min(k0 + CHUNK, K)):
            p = fx.fma(float(xr[k]), float(wr[k]), p)
        y = p if y is None else fx.add(y, p)
    return y


def check_f32w(L, seed=6):
    """FP32 weights: the FP32-weight probes (tests/golden/f32w_probes.json); every
    BF16 order probe with its weights widened to float32 (the same bits); exact
    rational emulation with full-precision weights; the binary64 bound; integer
    weights that bfloat16 cannot hold; and equality with the BF16 oracle when
    the weights are widened BF16 values."""
    fails = []
    for p in load_f32w_probes():
        x, w = f32w_probe_inputs(p)
        got = f32_bits(_linear_f32w(L, x, w)[0, 0])
        if got != int(p["expect_bits"], 16):
            fails.append(f"{p['name']}: got 0x{got:08x} want {p['expect_bits']}")
    for p in load_probes():
        x, wb = probe_inputs(p)
        w = (wb.astype(np.uint32) << 16).view(np.float32)
        got = f32_bits(_linear_f32w(L, x, w)[0, 0])
        if got != int(p["expect_bits"], 16):
            fails.append(f"{p['name']} with float32 weights: got 0x{got:08x} want {p['expect_bits']}")
    rng = np.random.default_rng(seed)
    for K in (1, 17, 256, 257, 520):
        x = rng.standard_normal((1, K)).astype(np.float32)
        w = (rng.standard_normal((1, K)) * 0.02).astype(np.float32)
        got = f32_bits(_linear_f32w(L, x, w)[0, 0])
        want = f32_bits(emulated_dot_f32w(x[0], w[0]))
        if got != want:
            fails.append(f"emulation K={K}: got 0x{got:08x} want 0x{want:08x}")
    K = 300
    x = (rng.standard_normal((1, K)) * 2.0 ** rng.integers(-70, 40, K)).astype(np.float32)
    w = (rng.standard_normal((1, K)) * 2.0 ** rng.integers(-120, 10, K)).astype(np.float32)
    if f32_bits(_linear_f32w(L, x, w)[0, 0]) != f32_bits(emulated_dot_f32w(x[0], w[0])):
        fails.append("emulation, wide range with subnormal weights")
    for K in (7, 255, 256, 257, 513, 1500, 4100):
        M, N = 2, 3
        x = rng.standard_normal((M, K)).astype(np.float32)
        w = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
        y = _linear_f32w(L, x, w).astype(np.float64)
        prod = x.astype(np.float64)[:, None, :] * w.astype(np.float64)[None, :, :]
        a = np.abs(prod).sum(axis=2)
        g64 = K * 2.0 ** -53 / (1 - K * 2.0 ** -53)
        if not np.all(np.abs(y - prod.sum(axis=2)) <= (gamma(K) + g64) * a):
            fails.append(f"binary64 bound K={K}")
    M, N, K = 3, 5, 1000
    xi = rng.integers(-3, 4, (M, K))
    wi = rng.integers(-300, 301, (N, K))        # most need more than bfloat16's 8 significant bits
    got = _linear_f32w(L, xi.astype(np.float32), wi.astype(np.float32))
    if not np.array_equal(got.astype(np.int64), xi @ wi.T) or not np.all(got == xi @ wi.T):
        fails.append("integer weights beyond bfloat16 precision are not exact")
    x = rng.standard_normal((4, 700)).astype(np.float32)
    wb = ((rng.standard_normal((6, 700)) * 0.02).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    y16 = _linear(_setup(L), x, wb)
    y32 = _linear_f32w(L, x, (wb.astype(np.uint32) << 16).view(np.float32))
    if not np.array_equal(y16.view(np.uint32), y32.view(np.uint32)):
        fails.append("widened BF16 weights as float32 differ from the BF16 path")
    return fails


ALL_CHECKS = {
    "probes": check_probes,
    "bias": check_bias,
    "f32w": check_f32w,
    "fp64_bound": check_fp64_bound,
    "integer_exact": check_integer_exact,
    "exact_emulation": check_exact_emulation,
    "invariants": check_invariants,
}
