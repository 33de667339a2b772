"""Binding of librg_probe.so (include/rg_probe.h): the read-bandwidth probe of the benchmark's floors.
Argument marshalling only."""
import ctypes
import os

import paper_2609_25624_amd as _rg

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librg_probe.so")
EXPORTS = ("rg_probe_read", "rg_probe_fma")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() (hipcc, gfx950)")
    L = ctypes.CDLL(LIB_PATH)
    L.rg_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p]
    L.rg_probe_read.restype = ctypes.c_int
    L.rg_probe_fma.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                               ctypes.c_void_p]
    L.rg_probe_fma.restype = ctypes.c_int
    return L


lib = _load()


def rg_probe_read(src, sink, grid, stream=None):
    """Read all of `src` (a device tensor; bytes a multiple of 8192); sink: uint32/int32 [grid * 256]."""
    import torch
    if not (isinstance(src, torch.Tensor) and src.is_cuda and src.is_contiguous()):
        raise TypeError("src must be a contiguous device tensor")
    if sink.numel() < grid * 256 or sink.element_size() != 4:
        raise ValueError("sink needs grid * 256 four-byte elements")
    rc = lib.rg_probe_read(src.data_ptr(), src.numel() * src.element_size(), sink.data_ptr(), int(grid),
                           _rg._stream_ptr(stream))
    if rc != 0:
        raise RuntimeError(f"rg_probe_read: status {rc}")


def rg_probe_fma(mode, chains, out, grid, iters, stream=None):
    """FMA issue-rate probe (mode 0 plain, 1 DPP row broadcast, 2 DPP quad broadcast, 3 SGPR operand,
    4 SGPR and plain operands in turn); out: float32 [grid * 256]."""
    import torch
    if not (isinstance(out, torch.Tensor) and out.is_cuda and out.dtype == torch.float32 and out.numel() >= grid * 256):
        raise ValueError("out must be a float32 device tensor of grid * 256 elements")
    rc = lib.rg_probe_fma(int(mode), int(chains), out.data_ptr(), int(grid), int(iters), _rg._stream_ptr(stream))
    if rc != 0:
        raise RuntimeError(f"rg_probe_fma: status {rc}")
