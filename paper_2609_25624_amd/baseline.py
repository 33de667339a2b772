"""Binding of librg_baseline.so (include/rg_baseline.h): the comparison point.

The scheme the fused layer replaces (Design, eq. 1): widen W into a transient
FP32 copy, then the vendor FP32 GEMM.  Used by the benchmark to time that
scheme through a C-ABI on the same buffers and stream.  Argument marshalling
only, as in the main binding.
"""
import ctypes
import os

import paper_2609_25624_amd as _rg

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librg_baseline.so")
EXPORTS = ("rg_linear_cast_baseline",)


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() (hipcc, gfx950)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64 = ctypes.c_void_p, ctypes.c_int64
    L.rg_linear_cast_baseline.argtypes = [vp, vp, vp, vp, i64, i64, i64, vp]
    L.rg_linear_cast_baseline.restype = ctypes.c_int
    return L


lib = _load()


def rg_linear_cast_baseline(x, w, w_tmp, y, stream=None):
    """y = x @ cast_f32(w).T through the transient FP32 copy w_tmp [N,K] and the vendor GEMM."""
    import torch
    px = _rg._tensor_ptr(x, (torch.float32,), "x")
    pw = _rg._tensor_ptr(w, (torch.bfloat16, torch.int16, torch.uint16), "w")
    pt = _rg._tensor_ptr(w_tmp, (torch.float32,), "w_tmp")
    py = _rg._tensor_ptr(y, (torch.float32,), "y")
    M, K = x.shape
    N = w.shape[0]
    if w.shape[1] != K or tuple(w_tmp.shape) != (N, K) or tuple(y.shape) != (M, N):
        raise ValueError(f"shapes x{tuple(x.shape)} w{tuple(w.shape)} w_tmp{tuple(w_tmp.shape)} y{tuple(y.shape)}")
    _rg._check(lib.rg_linear_cast_baseline(px, pw, pt, py, M, N, K, _rg._stream_ptr(stream)),
               "rg_linear_cast_baseline")
    return y
