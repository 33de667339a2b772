"""Binding of librg_negctl.so (include/rg_negctl.h): the negative controls.

Two linear layers that break the paper's design rules on purpose (an atomic
split-K and a split sized to the enabled compute units), used only by the
tests to show that the reproducibility checks catch what rg_linear avoids.
Argument marshalling only, as in the main binding.
"""
import ctypes
import os

import paper_2609_25624_amd as _rg

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librg_negctl.so")
RG_NEGCTL_OK, RG_NEGCTL_ERR_INVAL, RG_NEGCTL_ERR_HIP = 0, 1, 4
EXPORTS = ("rg_negctl_atomic_splitk", "rg_negctl_cu_split", "rg_negctl_last_hip_error")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() (hipcc, gfx950)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    L.rg_negctl_atomic_splitk.argtypes = [vp, vp, vp, i64, i64, i64, i32, vp]
    L.rg_negctl_cu_split.argtypes = [vp, vp, vp, i64, i64, i64, vp, ctypes.POINTER(i32)]
    L.rg_negctl_last_hip_error.argtypes = []
    for name in EXPORTS:
        getattr(L, name).restype = ctypes.c_int
    return L


lib = _load()


def _check(code, where):
    if code != RG_NEGCTL_OK:
        raise RuntimeError(f"{where}: status {code} (hipError {lib.rg_negctl_last_hip_error()})")


def _ptrs(x, w, y):
    import torch
    px = _rg._tensor_ptr(x, (torch.float32,), "x")
    pw = _rg._tensor_ptr(w, (torch.bfloat16, torch.int16, torch.uint16), "w")
    py = _rg._tensor_ptr(y, (torch.float32,), "y")
    M, K = x.shape
    N = w.shape[0]
    if w.shape[1] != K or tuple(y.shape) != (M, N):
        raise ValueError(f"shape mismatch x{tuple(x.shape)} w{tuple(w.shape)} y{tuple(y.shape)}")
    return px, pw, py, M, N, K


def atomic_splitk(x, w, y, splits, stream=None):
    px, pw, py, M, N, K = _ptrs(x, w, y)
    _check(lib.rg_negctl_atomic_splitk(px, pw, py, M, N, K, int(splits), _rg._stream_ptr(stream)),
           "rg_negctl_atomic_splitk")
    return y


def cu_split(x, w, y, stream=None):
    """Returns the split the CU count of `stream` produced."""
    px, pw, py, M, N, K = _ptrs(x, w, y)
    s = ctypes.c_int32(0)
    _check(lib.rg_negctl_cu_split(px, pw, py, M, N, K, _rg._stream_ptr(stream), ctypes.byref(s)),
           "rg_negctl_cu_split")
    return s.value
