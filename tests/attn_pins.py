"""Pins that tie the attention oracle (rg_attn_oracle.c) to things other than itself.

Every check takes a loaded oracle library (a ctypes CDLL exposing rg_exp1,
rg_exp1_array and rg_attn_oracle), so the same checks run against the real
oracle and against deliberately broken copies (tests/test_attn_oracle_mutants.py).
Each returns a list of failure strings (empty = pass).

  * EXP1 against its definition carried out in exact rational arithmetic
    (tests/fp32_exact.py), and against math.exp within 2 ulp;
  * hand-derived probes (tests/golden/attn_probes.json);
  * closed forms: one position gives its value row exactly; identical keys
    give the mean of the value rows, rounded once;
  * the whole order emulated in exact rationals on small inputs;
  * binary64 softmax within a tolerance derived from the arithmetic;
  * invariants: each sequence alone equals the batch, positions past the
    length are ignored, query heads of one group permute their outputs.
"""
import ctypes
import json
import math
import os
from fractions import Fraction

import numpy as np

from tests import fp32_exact as fx

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "attn_probes.json")
CHUNK = 256
L2E = float.fromhex("0x1.715476p+0")
LN2_HI = float.fromhex("0x1.62e4p-1")
LN2_LO = float.fromhex("0x1.7f7d1cp-20")


def _coef(i):
    return fx.to_f32(Fraction(1, math.factorial(i)))


COEF = [_coef(i) for i in range(8)]


def _setup(L):
    vp, i64, ci = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    L.rg_exp1.argtypes = [ctypes.c_float]
    L.rg_exp1.restype = ctypes.c_float
    L.rg_exp1_array.argtypes = [vp, vp, i64]
    L.rg_exp1_array.restype = None
    L.rg_attn_oracle.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, ctypes.c_float, vp, ci]
    L.rg_attn_oracle.restype = ci
    return L


def exp1_lib(L, u):
    u = np.ascontiguousarray(u, dtype=np.float32)
    out = np.empty_like(u)
    L.rg_exp1_array(u.ctypes.data, out.ctypes.data, u.size)
    return out


def attn_lib(L, q, kc, vc, lens, scale, nthreads=4):
    q = np.ascontiguousarray(q, dtype=np.float32)
    kc = np.ascontiguousarray(kc, dtype=np.uint16)
    vc = np.ascontiguousarray(vc, dtype=np.uint16)
    lens = np.ascontiguousarray(lens, dtype=np.int32)
    B, H, D = q.shape
    Hkv, Lmax = kc.shape[1], kc.shape[2]
    scratch = np.empty((nthreads, Lmax), dtype=np.float32)
    out = np.empty((B, H, D), dtype=np.float32)
    rc = L.rg_attn_oracle(q.ctypes.data, kc.ctypes.data, vc.ctypes.data, lens.ctypes.data, out.ctypes.data,
                          B, H, Hkv, Lmax, D, float(np.float32(scale)), scratch.ctypes.data, nthreads)
    assert rc == 0
    return out


# ---- exact-rational emulation of the definitions ----
def _mul(a, b):
    if a == 0 or b == 0:
        return math.copysign(0.0, math.copysign(1.0, a) * math.copysign(1.0, b))
    return fx.to_f32(Fraction(a) * Fraction(b))


def _sub(a, b):
    return fx.add(a, -b)


def _div(a, b):
    if a == 0:
        return math.copysign(0.0, math.copysign(1.0, a) * math.copysign(1.0, b))
    return fx.to_f32(Fraction(a) / Fraction(b))


def emulated_exp1(u):
    u = float(np.float32(u))
    if u < -87.0:
        return 0.0
    k = float(round(_mul(u, L2E)))          # Python's round: to nearest, ties to even
    r = fx.fma(-k, LN2_HI, u)
    r = fx.fma(-k, LN2_LO, r)
    p = COEF[7]
    for i in range(6, -1, -1):
        p = fx.fma(p, r, COEF[i])
    return _mul(p, 2.0 ** int(k))


def emulated_attn(q, kc, vc, lens, scale):
    """RG-ATTN-1 on exact rationals, one (b, h) at a time (small inputs only)."""
    B, H, D = q.shape
    Hkv, Lmax = kc.shape[1], kc.shape[2]
    group = H // Hkv
    up = lambda b: fx.bf16_to_float(int(b))
    scale = float(np.float32(scale))
    out = np.zeros((B, H, D), dtype=np.float32)
    for b in range(B):
        L = min(max(int(lens[b]), 0), Lmax)
        for h in range(H):
            g = h // group
            t = []
            for l in range(L):
                z = None
                for d0 in range(0, D, CHUNK):
                    p = 0.0
                    for d in range(d0, min(d0 + CHUNK, D)):
                        p = fx.fma(float(q[b, h, d]), up(kc[b, g, l, d]), p)
                    z = p if z is None else fx.add(z, p)
                t.append(_mul(z, scale))
            m = max(t) if t else -math.inf
            e = [emulated_exp1(_sub(tl, m)) for tl in t]
            S = None
            for l0 in range(0, L, CHUNK):
                s = 0.0
                for l in range(l0, min(l0 + CHUNK, L)):
                    s = fx.add(s, e[l])
                S = s if S is None else fx.add(S, s)
            for d in range(D):
                N = None
                for l0 in range(0, L, CHUNK):
                    n = 0.0
                    for l in range(l0, min(l0 + CHUNK, L)):
                        n = fx.fma(e[l], up(vc[b, g, l, d]), n)
                    N = n if N is None else fx.add(N, n)
                out[b, h, d] = _div(N, S)
    return out


def bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


# ---- checks ----
def check_exp_definition(L, seed=0):
    """EXP1 bits against the definition carried out in exact rationals."""
    L = _setup(L)
    rng = np.random.default_rng(seed)
    u = np.concatenate([
        np.array([0.0, -0.0, -1e-30, -1e-7, -0.25, -0.3465735, -0.3465736, -0.5, -1.0, -0.6931472, -2.0,
                  -10.0, -20.5, -50.0, -86.0, -86.99, -87.0, -87.0001, -100.0, -1e30], dtype=np.float32),
        -rng.exponential(3.0, 120).astype(np.float32),
        -rng.uniform(80, 87, 30).astype(np.float32),
        -rng.uniform(0, 1e-3, 20).astype(np.float32)])
    got = exp1_lib(L, u)
    fails = []
    for a, g in zip(u, got):
        want = emulated_exp1(float(a))
        if fx.float_bits(float(g)) != fx.float_bits(float(np.float32(want))):
            fails.append(f"EXP1({float(a)!r}): got {float(g)!r} want {want!r}")
    return fails


def check_exp_accuracy(L, seed=1):
    """EXP1 within 2 ulp of the true exponential over [-87, 0]; exact at 0; zero below -87."""
    L = _setup(L)
    rng = np.random.default_rng(seed)
    u = np.concatenate([-rng.uniform(0, 87, 60000), -rng.exponential(0.5, 20000)]).astype(np.float32)
    got = exp1_lib(L, u).astype(np.float64)
    ref = np.exp(u.astype(np.float64))
    ulp = np.maximum(np.spacing(ref.astype(np.float32)).astype(np.float64), 2.0 ** -149)
    err = np.abs(got - ref) / ulp
    fails = []
    if err.max() > 2.0:
        i = int(np.argmax(err))
        fails.append(f"EXP1({u[i]!r}) is {err[i]:.2f} ulp from exp")
    if exp1_lib(L, np.array([0.0], np.float32))[0] != 1.0:
        fails.append("EXP1(0) != 1")
    if np.any(exp1_lib(L, np.array([-87.01, -1000.0, -np.inf], np.float32)) != 0.0):
        fails.append("EXP1 below -87 is not +0")
    s = np.sort(u)
    if np.any(np.diff(exp1_lib(L, s)) < 0):
        fails.append("EXP1 is not monotone")
    return fails


def load_probes():
    with open(GOLDEN) as f:
        return json.load(f)["probes"]


def probe_inputs(p):
    Lp, D = p["L"], 8
    q = np.zeros((1, 1, D), np.float32)
    q[0, 0, 0] = 1.0
    kc = np.zeros((1, 1, Lp, D), np.uint16)
    kc[0, 0, :, 0] = 0xC300                        # -128: EXP1 gives +0
    for a, b in p["hot"]:
        kc[0, 0, a:b, 0] = 0x0000
    vc = np.zeros((1, 1, Lp, D), np.uint16)
    for a, b, v in p["v0"]:
        vc[0, 0, a:b, 0] = int(v, 16)
    return q, kc, vc, np.array([Lp], np.int32)


def check_probes(L):
    L = _setup(L)
    fails = []
    for p in load_probes():
        q, kc, vc, lens = probe_inputs(p)
        out = attn_lib(L, q, kc, vc, lens, 1.0)
        got = int(bits(out)[0, 0, 0])
        if got != int(p["expect_bits"], 16) or np.any(bits(out)[0, 0, 1:] != 0):
            fails.append(f"{p['name']}: got 0x{got:08x} want {p['expect_bits']}")
    return fails


def _rand_case(rng, B, H, Hkv, Lmax, D, lens, kstd=1.0):
    q = rng.standard_normal((B, H, D)).astype(np.float32)
    kf = (rng.standard_normal((B, Hkv, Lmax, D)) * kstd).astype(np.float32)
    vf = rng.standard_normal((B, Hkv, Lmax, D)).astype(np.float32)
    kc = (kf.view(np.uint32) >> 16).astype(np.uint16)
    vc = (vf.view(np.uint32) >> 16).astype(np.uint16)
    return q, kc, vc, np.array(lens, np.int32)


def check_closed_forms(L, seed=2):
    """One position: out is its value row exactly.  Identical keys: out = RN(sum of values / L)."""
    L = _setup(L)
    rng = np.random.default_rng(seed)
    fails = []
    q, kc, vc, _ = _rand_case(rng, 2, 4, 2, 40, 64, [1, 1])
    out = attn_lib(L, q, kc, vc, np.array([1, 1], np.int32), 0.125)
    want = np.repeat((vc[:, :, 0, :].astype(np.uint32) << 16).view(np.float32), 2, axis=1)
    if not np.array_equal(bits(out), bits(want)):
        fails.append("one position: out is not its value row")
    Lp, D = 700, 16
    q = rng.standard_normal((1, 1, D)).astype(np.float32)
    kc = np.tile(((rng.standard_normal(D).astype(np.float32).view(np.uint32)) >> 16).astype(np.uint16), (1, 1, Lp, 1))
    vi = rng.integers(-50, 51, (1, 1, Lp, D))
    vc = (vi.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    out = attn_lib(L, q, kc, vc, np.array([Lp], np.int32), 0.25)
    want = [fx.to_f32(Fraction(int(vi[0, 0, :, d].sum()), Lp)) for d in range(D)]
    if not np.array_equal(bits(out[0, 0]), bits(np.array(want, np.float32))):
        fails.append("identical keys: out is not the rounded mean of the values")
    return fails


def check_emulation(L, seed=3):
    """The whole order in exact rationals on small inputs (positions across segment boundaries)."""
    L = _setup(L)
    rng = np.random.default_rng(seed)
    q, kc, vc, lens = _rand_case(rng, 2, 4, 2, 300, 8, [300, 7], kstd=2.0)
    out = attn_lib(L, q, kc, vc, lens, 0.35355339)
    want = emulated_attn(q, kc, vc, lens, 0.35355339)
    if not np.array_equal(bits(out), bits(want)):
        bad = int(np.count_nonzero(bits(out) != bits(want)))
        return [f"{bad} outputs differ from the exact emulation"]
    return []


def check_fp64(L, seed=4):
    """Binary64 softmax(q k^T scale) v: |out - ref| <= 1e-4 * max|v| (a dropped or doubled
    position moves an output by about max|v| / L, above 1e-3 here)."""
    L = _setup(L)
    rng = np.random.default_rng(seed)
    lens = [1, 255, 256, 257, 700]
    q, kc, vc, lens = _rand_case(rng, 5, 4, 1, 700, 64, lens)
    scale = 0.125
    out = attn_lib(L, q, kc, vc, lens, scale).astype(np.float64)
    kf = (kc.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    vf = (vc.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    fails = []
    for b in range(5):
        Lb = int(lens[b])
        for h in range(4):
            t = kf[b, 0, :Lb] @ q[b, h].astype(np.float64) * scale
            w = np.exp(t - t.max())
            ref = (w @ vf[b, 0, :Lb]) / w.sum()
            if np.max(np.abs(out[b, h] - ref)) > 1e-4 * np.max(np.abs(vf[b, 0, :Lb])):
                fails.append(f"b={b} h={h} L={Lb}: {np.max(np.abs(out[b, h] - ref)):.2e} from binary64")
    return fails


def check_invariants(L, seed=5):
    """Each sequence alone equals the batch; positions past the length do not matter;
    permuting the query heads of a group permutes their outputs."""
    L = _setup(L)
    rng = np.random.default_rng(seed)
    q, kc, vc, lens = _rand_case(rng, 3, 6, 2, 400, 32, [400, 123, 257])
    out = attn_lib(L, q, kc, vc, lens, 0.2)
    fails = []
    for b in range(3):
        o1 = attn_lib(L, q[b:b + 1], kc[b:b + 1], vc[b:b + 1], lens[b:b + 1], 0.2)
        if not np.array_equal(bits(o1[0]), bits(out[b])):
            fails.append(f"sequence {b} alone differs from the batch")
    kc2, vc2 = kc.copy(), vc.copy()
    kc2[1, :, 123:] = 0x7F00                        # garbage (large) past the length
    vc2[1, :, 123:] = 0x4F00
    if not np.array_equal(bits(attn_lib(L, q, kc2, vc2, lens, 0.2)), bits(out)):
        fails.append("positions past the length changed the output")
    perm = np.array([2, 0, 1, 5, 3, 4])            # within the groups {0,1,2} and {3,4,5}
    if not np.array_equal(bits(attn_lib(L, q[:, perm], kc, vc, lens, 0.2)), bits(out[:, perm])):
        fails.append("permuting query heads of a group did not permute the outputs")
    return fails


ALL_CHECKS = {
    "exp_definition": check_exp_definition,
    "exp_accuracy": check_exp_accuracy,
    "probes": check_probes,
    "closed_forms": check_closed_forms,
    "emulation": check_emulation,
    "fp64": check_fp64,
    "invariants": check_invariants,
}
