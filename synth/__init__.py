"""Seeded synthetic inputs (host side), shared by the oracle tests and the GPU path.

Only input generation lives here: no part of the linear layer's arithmetic.
The C source documents the generator; this module marshals numpy buffers.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None

# Tensor ids keep the streams of different tensors of one workload apart.
TID_X = 1
TID_W = 2
TID_B = 3
TID_Q, TID_K, TID_V = 4, 6, 7


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = ctypes.CDLL(_build.LIB)
        i64, u64, dbl, vp = ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p
        L.rg_synth_splitmix64.argtypes = [u64, i64, vp]
        L.rg_synth_normal_f32.argtypes = [vp, i64, i64, u64, u64, dbl, dbl]
        L.rg_synth_normal_bf16.argtypes = [vp, i64, i64, u64, u64, dbl, dbl]
        for f in (L.rg_synth_splitmix64, L.rg_synth_normal_f32, L.rg_synth_normal_bf16):
            f.restype = None
        _lib = L
    return _lib


def splitmix64(start: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.uint64)
    lib().rg_synth_splitmix64(start, n, out.ctypes.data)
    return out


def normal_f32(rows: int, cols: int, seed: int, tensor_id: int, std: float = 1.0,
               mean: float = 0.0) -> np.ndarray:
    """float32 [rows, cols] ~ N(mean, std^2), counter based (row r depends only on r and cols)."""
    out = np.empty((rows, cols), dtype=np.float32)
    lib().rg_synth_normal_f32(out.ctypes.data, rows, cols, seed, tensor_id, mean, std)
    return out


def normal_bf16(rows: int, cols: int, seed: int, tensor_id: int, std: float = 0.02,
                mean: float = 0.0) -> np.ndarray:
    """bfloat16 bit patterns (uint16) [rows, cols] ~ N(mean, std^2), rounded to nearest even."""
    out = np.empty((rows, cols), dtype=np.uint16)
    lib().rg_synth_normal_bf16(out.ctypes.data, rows, cols, seed, tensor_id, mean, std)
    return out


def layer_inputs(M: int, N: int, K: int, seed: int = 0, w_std: float = 0.02, layer: int = 0):
    """x f32 [M,K] ~ N(0,1) and W bf16 bits [N,K] ~ N(0, w_std^2) for one linear layer.

    `layer` selects distinct streams for different layers of one workload.
    """
    x = normal_f32(M, K, seed, TID_X + 16 * layer, 1.0)
    w = normal_bf16(N, K, seed, TID_W + 16 * layer, w_std)
    return x, w


def layer_bias(N: int, seed: int = 0, std: float = 0.02, layer: int = 0) -> np.ndarray:
    """float32 bias [N] ~ N(0, std^2) for one layer (a row of the same counter-based stream)."""
    return normal_f32(1, N, seed, TID_B + 16 * layer, std)[0]


def attn_inputs(B: int, H: int, Hkv: int, Lmax: int, D: int, seed: int = 0, kstd: float = 1.0):
    """Decode attention inputs: q f32 [B,H,D] ~ N(0,1); key and value caches as bfloat16 bits
    [B,Hkv,Lmax,D], keys ~ N(0, kstd^2), values ~ N(0,1).  Row r of a cache is position r % Lmax
    of sequence-head r // Lmax, so a shorter Lmax is not a prefix; callers slice instead."""
    q = normal_f32(B * H, D, seed, TID_Q, 1.0).reshape(B, H, D)
    k = normal_bf16(B * Hkv * Lmax, D, seed, TID_K, kstd).reshape(B, Hkv, Lmax, D)
    v = normal_bf16(B * Hkv * Lmax, D, seed, TID_V, 1.0).reshape(B, Hkv, Lmax, D)
    return q, k, v
