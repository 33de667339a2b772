"""Thin Python binding of librg (include/rg.h): argument marshalling only.

Every step of the linear layer runs in the HIP kernels of librg.so; this
module passes device pointers, sizes and the stream through ctypes.  PyTorch
is used for device memory and streams only.  If librg.so is missing the
import fails loudly: there is no CPU fallback.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librg.so")

RG_OK, RG_ERR_INVAL, RG_ERR_ALIGN, RG_ERR_ARCH, RG_ERR_HIP, RG_ERR_RANGE, RG_ERR_ALIAS = range(7)
KERNELS = {0: "generic", 1: "decode", 2: "tiled", 3: "decode_xs", 4: "gemv", 5: "stream", 6: "ktile", 7: "skinny", 8: "wtile"}
CHUNK = 256


class RgError(RuntimeError):
    def __init__(self, code, where):
        self.code = code
        extra = ""
        if code == RG_ERR_HIP:
            extra = f", hipError {lib.rg_last_hip_error()}"
        super().__init__(f"{where}: {strerror(code)} (rg status {code}{extra})")


class rg_launch_t(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_int32), ("waves_per_wg", ctypes.c_int32), ("grid_wgs", ctypes.c_int32),
                ("depth", ctypes.c_int32), ("grid_order", ctypes.c_int32), ("tile_n", ctypes.c_int32),
                ("slice_m", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class rg_plan_t(ctypes.Structure):
    _fields_ = [("order_id", ctypes.c_int32), ("chunk", ctypes.c_int32), ("nchunks", ctypes.c_int64),
                ("kernel", ctypes.c_int32), ("waves_per_wg", ctypes.c_int32), ("grid_wgs", ctypes.c_int32),
                ("depth", ctypes.c_int32), ("rows_per_round", ctypes.c_int32), ("tile_m", ctypes.c_int32),
                ("tile_n", ctypes.c_int32)]


def _load():
    # librg.so needs libamdhip64.so.7.  PyTorch ships its own copy of the HIP
    # runtime; loading torch first makes the dynamic loader bind librg.so to
    # that same runtime (same soname), so device pointers and streams from
    # torch are valid in librg.  Two HIP runtimes in one process do not share
    # the device (the second reports no device).
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() (hipcc, gfx950)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    sig = {
        "rg_linear": [vp, vp, vp, i64, i64, i64, vp],
        "rg_linear_bias": [vp, vp, vp, vp, i64, i64, i64, vp],
        "rg_linear_f32w": [vp, vp, vp, i64, i64, i64, vp],
        "rg_linear_set_launch": [ctypes.POINTER(rg_launch_t)],
        "rg_plan": [i64, i64, i64, ctypes.POINTER(rg_plan_t)],
        "rg_plan_f32w": [i64, i64, i64, ctypes.POINTER(rg_plan_t)],
        "rg_cast_bf16_f32": [vp, vp, i64, vp],
        "rg_argmax_rows": [vp, vp, i64, i64, vp],
        "rg_stream_create_cu_mask": [ctypes.POINTER(ctypes.c_uint32), ctypes.c_uint32, ctypes.POINTER(vp)],
        "rg_stream_destroy": [vp],
        "rg_device_cu_count": [ctypes.POINTER(i32)],
        "rg_attn_decode": [vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, ctypes.c_float, vp, i64, vp],
        "rg_attn_decode_noalloc": [vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, ctypes.c_float, vp],
        "rg_strerror": [ctypes.c_int],
        "rg_last_hip_error": [],
    }
    for name, args in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    L.rg_strerror.restype = ctypes.c_char_p
    L.rg_attn_workspace_size.argtypes = [i64, i64, i64, i64]
    L.rg_attn_workspace_size.restype = i64
    return L


lib = _load()

# Every symbol include/rg.h declares (checked by the tests).
EXPORTS = ("rg_linear", "rg_linear_bias", "rg_linear_f32w", "rg_linear_set_launch", "rg_plan", "rg_plan_f32w",
           "rg_cast_bf16_f32", "rg_argmax_rows",
           "rg_stream_create_cu_mask", "rg_stream_destroy", "rg_device_cu_count", "rg_strerror",
           "rg_last_hip_error")
# ... and include/rg_attn.h.
ATTN_EXPORTS = ("rg_attn_workspace_size", "rg_attn_decode", "rg_attn_decode_noalloc")
ATTN_SCRATCH_BYTES = 64 << 20   # RG_ATTN_SCRATCH_BYTES


def strerror(code: int) -> str:
    return lib.rg_strerror(int(code)).decode()


def _check(code, where):
    if code != RG_OK:
        raise RgError(code, where)


def _stream_ptr(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _tensor_ptr(t, dtypes, name):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous (row-major)")
    cur = torch.cuda.current_device()
    if t.device.index != cur:
        # the library launches on the current device; memory of another device is not passed on
        raise ValueError(f"{name} is on {t.device} but the current device is cuda:{cur}")
    return t.data_ptr()


def rg_linear(x, w, y, stream=None):
    """y[M,N] = x[M,K] * up(w[N,K])^T in the fixed order (float32 x, y; bfloat16 w)."""
    import torch
    px = _tensor_ptr(x, (torch.float32,), "x")
    pw = _tensor_ptr(w, (torch.bfloat16, torch.int16, torch.uint16), "w")
    py = _tensor_ptr(y, (torch.float32,), "y")
    if x.dim() != 2 or w.dim() != 2 or y.dim() != 2:
        raise ValueError("x, w, y must be 2-D")
    M, K = x.shape
    N = w.shape[0]
    if w.shape[1] != K or tuple(y.shape) != (M, N):
        raise ValueError(f"shape mismatch x{tuple(x.shape)} w{tuple(w.shape)} y{tuple(y.shape)}")
    _check(lib.rg_linear(px, pw, py, M, N, K, _stream_ptr(stream)), "rg_linear")
    return y


def rg_linear_bias(x, w, b, y, stream=None):
    """y[M,N] = x[M,K] * up(w[N,K])^T + b[N]: the fixed-order product, then one add of b."""
    import torch
    px = _tensor_ptr(x, (torch.float32,), "x")
    pw = _tensor_ptr(w, (torch.bfloat16, torch.int16, torch.uint16), "w")
    pb = _tensor_ptr(b, (torch.float32,), "b")
    py = _tensor_ptr(y, (torch.float32,), "y")
    if x.dim() != 2 or w.dim() != 2 or y.dim() != 2 or b.dim() != 1:
        raise ValueError("x, w, y must be 2-D and b 1-D")
    M, K = x.shape
    N = w.shape[0]
    if w.shape[1] != K or tuple(y.shape) != (M, N) or b.shape[0] != N:
        raise ValueError(f"shape mismatch x{tuple(x.shape)} w{tuple(w.shape)} b{tuple(b.shape)} y{tuple(y.shape)}")
    _check(lib.rg_linear_bias(px, pw, pb, py, M, N, K, _stream_ptr(stream)), "rg_linear_bias")
    return y


def rg_linear_f32w(x, w, y, stream=None):
    """y[M,N] = x[M,K] * w[N,K]^T in the fixed order with float32 weights used as they are."""
    import torch
    px = _tensor_ptr(x, (torch.float32,), "x")
    pw = _tensor_ptr(w, (torch.float32,), "w")
    py = _tensor_ptr(y, (torch.float32,), "y")
    if x.dim() != 2 or w.dim() != 2 or y.dim() != 2:
        raise ValueError("x, w, y must be 2-D")
    M, K = x.shape
    N = w.shape[0]
    if w.shape[1] != K or tuple(y.shape) != (M, N):
        raise ValueError(f"shape mismatch x{tuple(x.shape)} w{tuple(w.shape)} y{tuple(y.shape)}")
    _check(lib.rg_linear_f32w(px, pw, py, M, N, K, _stream_ptr(stream)), "rg_linear_f32w")
    return y


def rg_linear_ptr(x_ptr, w_ptr, y_ptr, M, N, K, stream_ptr=0):
    """Raw-pointer form of rg_linear (device pointers as integers)."""
    _check(lib.rg_linear(x_ptr, w_ptr, y_ptr, M, N, K, stream_ptr), "rg_linear")


def rg_linear_set_launch(cfg=None, **kw):
    """Scheduling overrides (kernel, waves_per_wg, grid_wgs, depth, grid_order, tile_n, slice_m); None resets."""
    if cfg is None and not kw:
        _check(lib.rg_linear_set_launch(None), "rg_linear_set_launch")
        return
    c = rg_launch_t()
    for k, v in dict(cfg or {}, **kw).items():
        if k == "kernel" and isinstance(v, str):
            v = {n: i + 1 for i, n in KERNELS.items()}[v]
        setattr(c, k, int(v))
    _check(lib.rg_linear_set_launch(ctypes.byref(c)), "rg_linear_set_launch")


def rg_plan(M, N, K):
    p = rg_plan_t()
    _check(lib.rg_plan(M, N, K, ctypes.byref(p)), "rg_plan")
    d = {f: getattr(p, f) for f, _ in rg_plan_t._fields_}
    d["kernel_name"] = KERNELS.get(d["kernel"], "?")
    return d


def rg_plan_f32w(M, N, K):
    p = rg_plan_t()
    _check(lib.rg_plan_f32w(M, N, K, ctypes.byref(p)), "rg_plan_f32w")
    d = {f: getattr(p, f) for f, _ in rg_plan_t._fields_}
    d["kernel_name"] = KERNELS.get(d["kernel"], "?")
    return d


def rg_cast_bf16_f32(w, out, stream=None):
    import torch
    pw = _tensor_ptr(w, (torch.bfloat16, torch.int16, torch.uint16), "w")
    po = _tensor_ptr(out, (torch.float32,), "out")
    if out.numel() != w.numel():
        raise ValueError("out must have w.numel() elements")
    _check(lib.rg_cast_bf16_f32(pw, po, w.numel(), _stream_ptr(stream)), "rg_cast_bf16_f32")
    return out


def rg_argmax_rows(y, out, stream=None):
    import torch
    py = _tensor_ptr(y, (torch.float32,), "y")
    po = _tensor_ptr(out, (torch.int64,), "out")
    M, N = y.shape
    if out.numel() != M:
        raise ValueError("out must have one entry per row")
    _check(lib.rg_argmax_rows(py, po, M, N, _stream_ptr(stream)), "rg_argmax_rows")
    return out


def rg_stream_create_cu_mask(mask_words):
    arr = (ctypes.c_uint32 * len(mask_words))(*[int(m) & 0xFFFFFFFF for m in mask_words])
    s = ctypes.c_void_p()
    _check(lib.rg_stream_create_cu_mask(arr, len(mask_words), ctypes.byref(s)), "rg_stream_create_cu_mask")
    return s.value


def rg_stream_destroy(stream_ptr):
    _check(lib.rg_stream_destroy(stream_ptr), "rg_stream_destroy")


def rg_device_cu_count():
    n = ctypes.c_int32()
    _check(lib.rg_device_cu_count(ctypes.byref(n)), "rg_device_cu_count")
    return n.value


def rg_attn_workspace_size(B, H, Lmax, D):
    return int(lib.rg_attn_workspace_size(B, H, Lmax, D))


def rg_attn_decode(q, kc, vc, lens, out, scale, workspace=None, stream=None):
    """Fixed-order decode attention: q f32 [B,H,D], kc/vc bf16 [B,Hkv,Lmax,D], lens int32 [B], out f32 [B,H,D].
    `workspace` (a uint8 device tensor of rg_attn_workspace_size bytes) is allocated by torch if None."""
    import torch
    pq = _tensor_ptr(q, (torch.float32,), "q")
    pk = _tensor_ptr(kc, (torch.bfloat16, torch.int16, torch.uint16), "kc")
    pv = _tensor_ptr(vc, (torch.bfloat16, torch.int16, torch.uint16), "vc")
    pl = _tensor_ptr(lens, (torch.int32,), "lens")
    po = _tensor_ptr(out, (torch.float32,), "out")
    if q.dim() != 3 or kc.dim() != 4 or tuple(vc.shape) != tuple(kc.shape) or tuple(out.shape) != tuple(q.shape):
        raise ValueError("q/out [B,H,D], kc/vc [B,Hkv,Lmax,D]")
    B, H, D = q.shape
    _, Hkv, Lmax, D2 = kc.shape
    if kc.shape[0] != B or D2 != D or lens.numel() != B:
        raise ValueError(f"shape mismatch q{tuple(q.shape)} kc{tuple(kc.shape)} lens{tuple(lens.shape)}")
    need = rg_attn_workspace_size(B, H, Lmax, D)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    pw = _tensor_ptr(workspace, (torch.uint8,), "workspace")
    _check(lib.rg_attn_decode(pq, pk, pv, pl, po, B, H, Hkv, Lmax, D, float(scale), pw, workspace.numel(),
                              _stream_ptr(stream)), "rg_attn_decode")
    return out


def rg_attn_decode_noalloc(q, kc, vc, lens, out, scale, stream=None):
    """rg_attn_decode with the library's static device scratch as workspace (allocates nothing;
    workspaces beyond ATTN_SCRATCH_BYTES are refused with RG_ERR_RANGE).  Calls that overlap in
    time on one device share that scratch and race."""
    import torch
    pq = _tensor_ptr(q, (torch.float32,), "q")
    pk = _tensor_ptr(kc, (torch.bfloat16, torch.int16, torch.uint16), "kc")
    pv = _tensor_ptr(vc, (torch.bfloat16, torch.int16, torch.uint16), "vc")
    pl = _tensor_ptr(lens, (torch.int32,), "lens")
    po = _tensor_ptr(out, (torch.float32,), "out")
    if q.dim() != 3 or kc.dim() != 4 or tuple(vc.shape) != tuple(kc.shape) or tuple(out.shape) != tuple(q.shape):
        raise ValueError("q/out [B,H,D], kc/vc [B,Hkv,Lmax,D]")
    B, H, D = q.shape
    _, Hkv, Lmax, D2 = kc.shape
    if kc.shape[0] != B or D2 != D or lens.numel() != B:
        raise ValueError(f"shape mismatch q{tuple(q.shape)} kc{tuple(kc.shape)} lens{tuple(lens.shape)}")
    _check(lib.rg_attn_decode_noalloc(pq, pk, pv, pl, po, B, H, Hkv, Lmax, D, float(scale), _stream_ptr(stream)),
           "rg_attn_decode_noalloc")
    return out
