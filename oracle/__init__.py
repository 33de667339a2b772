"""CPU oracle of the fused-upcast linear layer (ctypes wrapper over rg_oracle.c).

TEST INFRASTRUCTURE ONLY.  Only tests/, the smoke check and the benchmark's
CPU-baseline leg may import this package; the GPU path never does.  The order
it computes is documented at the top of rg_oracle.c.
"""
import ctypes
import os

import numpy as np

from . import build as _build

CHUNK = 256
U32 = 2.0 ** -24  # unit roundoff of binary32, round to nearest

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = ctypes.CDLL(_build.LIB)
        i64, vp, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
        L.rg_oracle_dot.argtypes = [vp, vp, i64]
        L.rg_oracle_dot.restype = ctypes.c_float
        L.rg_oracle_linear.argtypes = [vp, vp, vp, i64, i64, i64, ci]
        L.rg_oracle_linear.restype = ci
        L.rg_oracle_linear_bias.argtypes = [vp, vp, vp, vp, i64, i64, i64, ci]
        L.rg_oracle_linear_bias.restype = ci
        L.rg_oracle_linear_f32w.argtypes = [vp, vp, vp, i64, i64, i64, ci]
        L.rg_oracle_linear_f32w.restype = ci
        L.rg_ref_fp64_f32w.argtypes = [vp, vp, vp, vp, i64, i64, i64, ci]
        L.rg_ref_fp64_f32w.restype = ci
        L.rg_oracle_linear_sampled.argtypes = [vp, vp, i64, vp, vp, i64, vp, ci]
        L.rg_oracle_linear_sampled.restype = ci
        L.rg_ref_fp64.argtypes = [vp, vp, vp, vp, i64, i64, i64, ci]
        L.rg_ref_fp64.restype = ci
        L.rg_exp1.argtypes = [ctypes.c_float]
        L.rg_exp1.restype = ctypes.c_float
        L.rg_exp1_array.argtypes = [vp, vp, i64]
        L.rg_exp1_array.restype = None
        L.rg_attn_oracle.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, ctypes.c_float, vp, ci]
        L.rg_attn_oracle.restype = ci
        L.rg_oracle_argmax.argtypes = [vp, i64]
        L.rg_oracle_argmax.restype = i64
        L.rg_oracle_fast_linear.argtypes = [vp, vp, vp, i64, i64, i64, ci]
        L.rg_oracle_fast_linear.restype = ci
        L.rg_oracle_fast_supported.argtypes = []
        L.rg_oracle_fast_supported.restype = ci
        _lib = L
    return _lib


def _threads(nthreads):
    if nthreads:
        return int(nthreads)
    return int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))


def _check(x, w):
    x = np.ascontiguousarray(x, dtype=np.float32)
    w = np.ascontiguousarray(w)
    if w.dtype != np.uint16:
        raise TypeError("w must hold bfloat16 bit patterns as uint16")
    if x.ndim != 2 or w.ndim != 2 or x.shape[1] != w.shape[1]:
        raise ValueError(f"shape mismatch x{x.shape} w{w.shape}")
    return x, w


def linear(x, w, nthreads=None) -> np.ndarray:
    """y[M,N] (float32) in the documented order, x f32 [M,K], w bf16 bits [N,K]."""
    x, w = _check(x, w)
    M, K = x.shape
    N = w.shape[0]
    y = np.empty((M, N), dtype=np.float32)
    rc = lib().rg_oracle_linear(x.ctypes.data, w.ctypes.data, y.ctypes.data, M, N, K, _threads(nthreads))
    if rc != 0:
        raise ValueError("rg_oracle_linear rejected its arguments")
    return y


def fast_supported() -> bool:
    """Whether this CPU runs the same-order vectorised oracle (AVX2 and FMA)."""
    return bool(lib().rg_oracle_fast_supported())


def linear_fast(x, w, nthreads=None) -> np.ndarray:
    """linear() computed by the same-order vectorised oracle (rg_oracle_fast.c): the same operation
    sequence per output, sixteen outputs per AVX2 register pair; bit-identical to linear() (pinned
    by the tests).  For the largest workloads."""
    x, w = _check(x, w)
    M, K = x.shape
    N = w.shape[0]
    y = np.empty((M, N), dtype=np.float32)
    rc = lib().rg_oracle_fast_linear(x.ctypes.data, w.ctypes.data, y.ctypes.data, M, N, K, _threads(nthreads))
    if rc == -2:
        raise RuntimeError("the same-order vectorised oracle needs AVX2 and FMA on the host CPU")
    if rc != 0:
        raise ValueError(f"rg_oracle_fast_linear failed ({rc})")
    return y


def linear_f32w(x, w, nthreads=None) -> np.ndarray:
    """y[M,N] in the documented order with float32 weights w [N,K] used as they are."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    w = np.ascontiguousarray(w)
    if w.dtype != np.float32:
        raise TypeError("w must be float32")
    if x.ndim != 2 or w.ndim != 2 or x.shape[1] != w.shape[1]:
        raise ValueError(f"shape mismatch x{x.shape} w{w.shape}")
    M, K = x.shape
    N = w.shape[0]
    y = np.empty((M, N), dtype=np.float32)
    rc = lib().rg_oracle_linear_f32w(x.ctypes.data, w.ctypes.data, y.ctypes.data, M, N, K, _threads(nthreads))
    if rc != 0:
        raise ValueError("rg_oracle_linear_f32w rejected its arguments")
    return y


def linear_bias(x, w, b, nthreads=None) -> np.ndarray:
    """y[M,N] = (the documented order) + b[N], one binary32 addition after the fold."""
    x, w = _check(x, w)
    b = np.ascontiguousarray(b, dtype=np.float32)
    M, K = x.shape
    N = w.shape[0]
    if b.shape != (N,):
        raise ValueError(f"bias shape {b.shape}, expected ({N},)")
    y = np.empty((M, N), dtype=np.float32)
    rc = lib().rg_oracle_linear_bias(x.ctypes.data, w.ctypes.data, b.ctypes.data, y.ctypes.data, M, N, K,
                                     _threads(nthreads))
    if rc != 0:
        raise ValueError("rg_oracle_linear_bias rejected its arguments")
    return y


def linear_sampled(x, w, rows, cols, nthreads=None) -> np.ndarray:
    """out[s] = y[rows[s], cols[s]] without computing the rest of y."""
    x, w = _check(x, w)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    if rows.shape != cols.shape:
        raise ValueError("rows/cols length mismatch")
    if rows.size and (rows.min() < 0 or rows.max() >= x.shape[0] or cols.min() < 0 or cols.max() >= w.shape[0]):
        raise IndexError("sample index out of range")
    out = np.empty(rows.shape, dtype=np.float32)
    rc = lib().rg_oracle_linear_sampled(x.ctypes.data, w.ctypes.data, x.shape[1], rows.ctypes.data,
                                        cols.ctypes.data, rows.size, out.ctypes.data, _threads(nthreads))
    if rc != 0:
        raise ValueError("rg_oracle_linear_sampled rejected its arguments")
    return out


def dot(x_row, w_row) -> np.float32:
    x_row = np.ascontiguousarray(x_row, dtype=np.float32).ravel()
    w_row = np.ascontiguousarray(w_row, dtype=np.uint16).ravel()
    if x_row.size != w_row.size or x_row.size < 1:
        raise ValueError("dot needs two rows of equal positive length")
    return np.float32(lib().rg_oracle_dot(x_row.ctypes.data, w_row.ctypes.data, x_row.size))


def ref_fp64(x, w, nthreads=None):
    """(y64, abs_sum): the sum in binary64 and the sum of |x*w| per output."""
    x, w = _check(x, w)
    M, K = x.shape
    N = w.shape[0]
    y64 = np.empty((M, N), dtype=np.float64)
    a = np.empty((M, N), dtype=np.float64)
    rc = lib().rg_ref_fp64(x.ctypes.data, w.ctypes.data, y64.ctypes.data, a.ctypes.data, M, N, K,
                           _threads(nthreads))
    if rc != 0:
        raise ValueError("rg_ref_fp64 rejected its arguments")
    return y64, a


def gamma(K: int) -> float:
    """Error bound factor gamma_n, n = longest rounding path = min(C,K) + J - 1."""
    J = -(-K // CHUNK)
    n = min(CHUNK, K) + J - 1
    return n * U32 / (1.0 - n * U32)


def argmax(v) -> int:
    v = np.ascontiguousarray(v, dtype=np.float32).ravel()
    return int(lib().rg_oracle_argmax(v.ctypes.data, v.size))


def exp1(u) -> np.ndarray:
    """EXP1 (the exponential of the fixed-order attention) elementwise on float32 input."""
    u = np.ascontiguousarray(u, dtype=np.float32)
    out = np.empty_like(u)
    lib().rg_exp1_array(u.ctypes.data, out.ctypes.data, u.size)
    return out


def attn_decode(q, kc, vc, lens, scale, nthreads=None) -> np.ndarray:
    """Fixed-order decode attention: q f32 [B,H,D], kc/vc bf16 bits [B,Hkv,Lmax,D], lens int32 [B]."""
    q = np.ascontiguousarray(q, dtype=np.float32)
    kc = np.ascontiguousarray(kc)
    vc = np.ascontiguousarray(vc)
    if kc.dtype != np.uint16 or vc.dtype != np.uint16:
        raise TypeError("kc and vc must hold bfloat16 bit patterns as uint16")
    lens = np.ascontiguousarray(lens, dtype=np.int32)
    B, H, D = q.shape
    _, Hkv, Lmax, D2 = kc.shape
    if kc.shape != vc.shape or kc.shape[0] != B or D2 != D or lens.shape != (B,):
        raise ValueError("shape mismatch")
    nt = _threads(nthreads)
    scratch = np.empty((nt, Lmax), dtype=np.float32)
    out = np.empty((B, H, D), dtype=np.float32)
    rc = lib().rg_attn_oracle(q.ctypes.data, kc.ctypes.data, vc.ctypes.data, lens.ctypes.data, out.ctypes.data,
                              B, H, Hkv, Lmax, D, float(np.float32(scale)), scratch.ctypes.data, nt)
    if rc != 0:
        raise ValueError("rg_attn_oracle rejected its arguments")
    return out
