"""The C-ABI library without a GPU: symbols, the shape-only planner, host-side argument checks."""
import ctypes
import os
import re

import pytest

import paper_2609_25624_amd as rg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rg.h")


_ASM_CACHE = {}


def _device_asm(fname):
    """gfx950 assembly of one of the library's sources, compiled once per test session."""
    if fname not in _ASM_CACHE:
        import subprocess
        import tempfile
        from paper_2609_25624_amd import build as b
        src = os.path.join(ROOT, "paper_2609_25624_amd", "csrc", fname)
        with tempfile.TemporaryDirectory() as d:
            out = os.path.join(d, "k.s")
            r = subprocess.run([b.HIPCC, "-x", "hip", *b.COMMON, *b.DEVICE, "--cuda-device-only", "-S", src, "-o", out],
                               capture_output=True, text=True)
            assert r.returncode == 0, r.stderr
            _ASM_CACHE[fname] = open(out).read()
    return _ASM_CACHE[fname]


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(rg_\w+)\s*\(", text, flags=re.M)))


def test_every_declared_symbol_is_exported_and_bound():
    names = declared_functions()
    assert "rg_linear" in names and "rg_linear_set_launch" in names
    lib = ctypes.CDLL(rg.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in include/rg.h but not exported"
    assert sorted(rg.EXPORTS) == names


def test_strerror_never_null():
    for c in range(-2, 10):
        assert isinstance(rg.strerror(c), str) and rg.strerror(c)


def test_plan_numeric_fields_depend_on_k_only():
    # The order (segment length, segment count, order id) is a function of K alone.
    for K in (1, 7, 8, 255, 256, 257, 1000, 4096, 14336, 28672):
        seen = set()
        for M in (1, 2, 4, 5, 16, 64, 65, 2048):
            for N in (1, 5, 1024, 4096, 128256):
                p = rg.rg_plan(M, N, K)
                seen.add((p["order_id"], p["chunk"], p["nchunks"]))
        assert seen == {(1, 256, -(-K // 256))}


def test_plan_is_pure_and_overrides_are_scheduling_only():
    for shape, ov in (((4, 6144, 4096), (4, 100, 2)), ((1, 6144, 4096), (2, 100, 3))):
        want = ov
        a = rg.rg_plan(*shape)
        assert a == rg.rg_plan(*shape)
        rg.rg_linear_set_launch(waves_per_wg=ov[0], grid_wgs=ov[1], depth=ov[2], grid_order=1)
        try:
            b = rg.rg_plan(*shape)
            assert (b["waves_per_wg"], b["grid_wgs"], b["depth"]) == want
            assert (b["order_id"], b["chunk"], b["nchunks"]) == (a["order_id"], a["chunk"], a["nchunks"])
            assert b["kernel"] == a["kernel"]
        finally:
            rg.rg_linear_set_launch(None)
        assert rg.rg_plan(*shape) == a


def test_gemv_schedule_defaults():
    # fewest rounds of quads per wave, then the fewest waves giving them, over all 256 workgroups
    rg.rg_linear_set_launch(kernel="gemv")
    try:
        p = rg.rg_plan(1, 4096, 4096)
        assert (p["kernel_name"], p["grid_wgs"], p["waves_per_wg"]) == ("gemv", 256, 4)
        p = rg.rg_plan(1, 6144, 4096)            # 1536 quads: two rounds of 768 waves
        assert (p["grid_wgs"], p["waves_per_wg"]) == (256, 3)
        p = rg.rg_plan(1, 28672, 4096)           # 7168 quads: seven rounds of 1024 waves
        assert (p["grid_wgs"], p["waves_per_wg"]) == (256, 4)
        p = rg.rg_plan(1, 4096, 14336)           # x staged a step at a time: four slots fit at any K
        assert (p["grid_wgs"], p["waves_per_wg"]) == (256, 4)
        p = rg.rg_plan(1, 3072, 8192)            # 768 quads: 3 waves would do, K > 4096 takes 4
        assert (p["grid_wgs"], p["waves_per_wg"]) == (192, 4)
    finally:
        rg.rg_linear_set_launch(None)
    rg.rg_linear_set_launch(kernel="gemv", waves_per_wg=3)
    try:
        with pytest.raises(rg.RgError):
            rg.rg_plan(1, 4096, 14336)           # K > 4096: the waves share the x part in 1, 2 or 4 shares
        assert rg.rg_plan(1, 4096, 4096)["waves_per_wg"] == 3
    finally:
        rg.rg_linear_set_launch(None)
    rg.rg_linear_set_launch(waves_per_wg=4)     # not forced: the planner's kernel takes the override
    try:
        assert rg.rg_plan(1, 4096, 14336)["kernel_name"] == "skinny"
    finally:
        rg.rg_linear_set_launch(None)


def test_skinny_slice_width():
    # where the row groups cap the walkers below the workgroups the CUs hold, the planner halves
    # the slice of x rows while that gives more workgroups; elsewhere the widest slice that fits
    want = {(1, 6144, 4096): 1, (2, 6144, 4096): 1, (2, 4096, 4096): 1, (3, 6144, 4096): 2,
            (4, 6144, 4096): 2, (4, 4096, 4096): 2, (4, 28672, 4096): 4, (4, 4096, 14336): 4,
            (4, 128256, 4096): 4, (8, 6144, 4096): 4, (16, 6144, 4096): 8, (16, 28672, 4096): 8,
            (16, 4096, 14336): 4}
    for shape, mt in want.items():
        p = rg.rg_plan(*shape)
        assert (p["kernel_name"], p["tile_m"]) == ("skinny", mt), (shape, p)
        assert p["grid_wgs"] <= 512
    with pytest.raises(rg.RgError):
        rg.rg_linear_set_launch(slice_m=3)
    try:
        rg.rg_linear_set_launch(kernel="skinny", slice_m=8)
        assert rg.rg_plan(4, 4096, 14336)["tile_m"] == 4      # two segment groups per wave: 4 rows fit
        assert rg.rg_plan(4, 6144, 4096)["tile_m"] == 8       # a slice wider than M is allowed
        rg.rg_linear_set_launch(slice_m=2)                      # not forced: applies where skinny runs
        p = rg.rg_plan(16, 28672, 4096)
        assert (p["kernel_name"], p["tile_m"], p["grid_wgs"]) == ("skinny", 2, 512)
        assert rg.rg_plan(64, 28672, 4096)["kernel_name"] == "ktile"
    finally:
        rg.rg_linear_set_launch(None)


def test_one_row_kernel_choice():
    # M = 1: the GEMV for K = 4096 on layers of at most 4096 rows, the skinny kernel elsewhere
    for shape, name in (((1, 4096, 4096), "gemv"), ((1, 2048, 4096), "gemv"), ((1, 6144, 4096), "skinny"),
                        ((1, 28672, 4096), "skinny"), ((1, 4096, 14336), "skinny"), ((1, 4096, 8192), "skinny"),
                        ((1, 1024, 1024), "skinny"), ((2, 4096, 4096), "skinny")):
        assert rg.rg_plan(*shape)["kernel_name"] == name, shape


def test_mid_batch_kernel_choice():
    # 16 < M <= 64: skinny on layers with fewer than 448 tiles of 64 W rows and K <= 16384, the
    # wave-tile kernel above M = 32 with 448 to 1024 such tiles, ktile elsewhere
    for shape, name in (((32, 6144, 4096), "skinny"), ((64, 4096, 4096), "skinny"), ((64, 4096, 14336), "skinny"),
                        ((17, 300, 1000), "skinny"), ((32, 28672, 4096), "ktile"), ((64, 128256, 4096), "ktile"),
                        ((33, 28672, 4096), "wtile"), ((64, 28672, 4096), "wtile"), ((64, 57344, 8192), "wtile"),
                        ((64, 8192, 28672), "ktile"), ((17, 4096, 16640), "ktile"), ((65, 4096, 4096), "tiled")):
        assert rg.rg_plan(*shape)["kernel_name"] == name, shape
    rg.rg_linear_set_launch(tile_n=32)          # not forced, not a wave-tile setting: ktile takes it
    try:
        p = rg.rg_plan(64, 28672, 4096)
        assert (p["kernel_name"], p["tile_n"]) == ("ktile", 32)
    finally:
        rg.rg_linear_set_launch(None)


def test_tiled_128_build_choice():
    # three waves per SIMD only where its rounds of 768 resident tiles are clearly fuller than
    # the two-wave build's rounds of 512; other tiles report depth 0
    cases = {(2048, 8192, 8192): 2,     # 1024 tiles: 2 full rounds of 512, 1.33 rounds of 768
             (2048, 57344, 8192): 2,    # 7168 tiles: 14 full rounds of 512
             (2048, 4096, 4096): 2,     # 512 tiles: one round either way
             (1100, 9000, 4096): 3}     # 639 tiles: 0.62 of two rounds of 512, 0.83 of one of 768
    for shape, depth in cases.items():
        p = rg.rg_plan(*shape)
        assert (p["kernel_name"], p["tile_m"], p["depth"]) == ("tiled", 128, depth), (shape, p)
    assert rg.rg_plan(256, 28672, 4096)["depth"] == 0          # 64 x 128 tiles
    rg.rg_linear_set_launch(depth=3)
    try:
        assert rg.rg_plan(2048, 8192, 8192)["depth"] == 3
    finally:
        rg.rg_linear_set_launch(None)


def test_set_launch_range_checks():
    for bad in (dict(waves_per_wg=9), dict(grid_wgs=-1), dict(depth=4), dict(depth=1), dict(grid_order=2), dict(kernel=10), dict(tile_n=48)):
        with pytest.raises(rg.RgError) as e:
            rg.rg_linear_set_launch(**bad)
        assert e.value.code == rg.RG_ERR_RANGE
    rg.rg_linear_set_launch(None)


def test_linear_rejects_bad_arguments_before_touching_a_device():
    L = rg.lib
    # null pointers, bad sizes, overflow
    assert L.rg_linear(None, 16, 16, 1, 1, 1, None) == rg.RG_ERR_INVAL
    assert L.rg_linear(16, 16, 1024, 0, 1, 1, None) == rg.RG_ERR_INVAL
    assert L.rg_linear(16, 16, 1024, 1, -3, 1, None) == rg.RG_ERR_INVAL
    assert L.rg_linear(16, 16, 1024, 1 << 40, 1, 1 << 30, None) == rg.RG_ERR_INVAL
    # misaligned x (4), W (2), y (4)
    assert L.rg_linear(0x1002, 0x100000, 0x200000, 1, 1, 8, None) == rg.RG_ERR_ALIGN
    assert L.rg_linear(0x1000, 0x100001, 0x200000, 1, 1, 8, None) == rg.RG_ERR_ALIGN
    assert L.rg_linear(0x1000, 0x100000, 0x200002, 1, 1, 8, None) == rg.RG_ERR_ALIGN
    # y overlapping x or W
    assert L.rg_linear(0x1000, 0x100000, 0x1000, 1, 1, 8, None) == rg.RG_ERR_ALIAS
    assert L.rg_linear(0x1000, 0x100000, 0x100008, 1, 2, 8, None) == rg.RG_ERR_ALIAS
    assert L.rg_plan(0, 1, 1, None) == rg.RG_ERR_INVAL


def test_other_entry_points_reject_bad_arguments():
    L = rg.lib
    assert L.rg_cast_bf16_f32(None, 0x1000, 10, None) == rg.RG_ERR_INVAL
    assert L.rg_cast_bf16_f32(0x1001, 0x1000, 10, None) == rg.RG_ERR_ALIGN
    assert L.rg_argmax_rows(0x1000, None, 1, 1, None) == rg.RG_ERR_INVAL
    assert L.rg_argmax_rows(0x1002, 0x2000, 1, 1, None) == rg.RG_ERR_ALIGN
    # overflow of the sizes, and an output overlapping its input
    assert L.rg_cast_bf16_f32(0x1000, 0x100000, 1 << 62, None) == rg.RG_ERR_INVAL
    assert L.rg_cast_bf16_f32(0x1000, 0x1010, 16, None) == rg.RG_ERR_ALIAS
    assert L.rg_argmax_rows(0x1000, 0x2000, 1 << 30, 1 << 40, None) == rg.RG_ERR_INVAL
    assert L.rg_argmax_rows(0x1000, 0x1008, 2, 4, None) == rg.RG_ERR_ALIAS
    assert L.rg_argmax_rows(0x1000, 0x1000 - 8, 2, 4, None) == rg.RG_ERR_ALIAS
    assert L.rg_stream_create_cu_mask(None, 1, None) == rg.RG_ERR_INVAL
    assert L.rg_stream_destroy(None) == rg.RG_ERR_INVAL
    assert L.rg_device_cu_count(None) == rg.RG_ERR_INVAL


@pytest.mark.parametrize("fname", ["rg_kernels.hip", "rg_wtile.hip"])
def test_no_atomics_or_matrix_core_builtins_in_kernels(fname):
    src = open(os.path.join(ROOT, "paper_2609_25624_amd", "csrc", fname)).read()
    code = re.sub(r"//.*", "", src)
    for bad in ("atomicAdd", "__hip_atomic", "mfma", "__builtin_amdgcn_fdot", "__builtin_amdgcn_sdot",
                "unsafe-fp", "fast-math"):
        assert bad not in code, bad


@pytest.mark.parametrize("fname", ["rg_kernels.hip", "rg_wtile.hip"])
def test_device_code_uses_only_ieee_fma_for_accumulation(fname):
    # Inspect the gfx950 assembly of our own kernels: no matrix-core, dot-product,
    # packed-FP32, mixed-precision or non-fused multiply-add instructions.
    asm = _device_asm(fname)
    insts = re.findall(r"^\s+(v_[a-z0-9_]+)", asm, flags=re.M)
    assert insts
    for i in set(insts):
        assert not re.match(r"v_(mfma|smfmac|dot\d|pk_(fma|mul|add)_f32|mad_f32|mac_f32|mad_legacy|mac_legacy|fma_legacy|fma_mix|mad_mix)", i), i
    assert "v_fma_f32" in insts or "v_fmac_f32_e32" in insts
    # binary32 denormals kept in every kernel
    modes = re.findall(r"\.amdhsa_float_denorm_mode_32\s+(\d+)", asm)
    assert modes and set(modes) == {"3"}


def test_negative_control_library_exports_its_header_and_checks_arguments():
    # The negative controls live in a library of their own; rg_linear's library holds none of them.
    from paper_2609_25624_amd import negctl
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "rg_negctl.h")).read(), flags=re.S)
    names = sorted(set(re.findall(r"^\s*int\s+(rg_negctl_\w+)\s*\(", text, flags=re.M)))
    assert sorted(negctl.EXPORTS) == names
    lib = ctypes.CDLL(negctl.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    main = ctypes.CDLL(rg.LIB_PATH)
    for n in names:
        assert not hasattr(main, n), f"{n} must not be in librg.so"
    L = negctl.lib
    assert L.rg_negctl_atomic_splitk(None, 0x1000, 0x2000, 1, 1, 8, 2, None) == negctl.RG_NEGCTL_ERR_INVAL
    assert L.rg_negctl_atomic_splitk(0x1000, 0x2000, 0x3000, 1, 1, 8, 0, None) == negctl.RG_NEGCTL_ERR_INVAL
    assert L.rg_negctl_atomic_splitk(0x1000, 0x2000, 0x3000, 1, 1, 8, 9, None) == negctl.RG_NEGCTL_ERR_INVAL
    assert L.rg_negctl_atomic_splitk(0x1002, 0x2000, 0x3000, 1, 1, 8, 2, None) == negctl.RG_NEGCTL_ERR_INVAL
    assert L.rg_negctl_cu_split(0x1000, 0x2000, 0x3000, 0, 1, 8, None, None) == negctl.RG_NEGCTL_ERR_INVAL
    assert L.rg_negctl_cu_split(0x1000, 0x2001, 0x3000, 1, 1, 8, None, None) == negctl.RG_NEGCTL_ERR_INVAL


def test_f32w_planner_and_argument_checks():
    rg.rg_linear_set_launch(None)
    assert rg.rg_plan_f32w(1, 4096, 14336)["kernel_name"] == "stream"
    assert rg.rg_plan_f32w(4, 6144, 4096)["kernel_name"] == "stream"
    assert rg.rg_plan_f32w(16, 6144, 4096)["kernel_name"] == "ktile"
    assert rg.rg_plan_f32w(100, 1000, 1000)["kernel_name"] == "tiled"
    assert rg.rg_plan_f32w(1, 100, 1001)["kernel_name"] == "generic"      # K % 4 != 0
    assert rg.rg_plan_f32w(1, 4096, 4100)["nchunks"] == 17
    try:
        for k in ("decode", "decode_xs", "gemv"):
            rg.rg_linear_set_launch(kernel=k)
            with pytest.raises(rg.RgError):
                rg.rg_plan_f32w(1, 4096, 4096)
        rg.rg_linear_set_launch(kernel="stream")
        assert rg.rg_plan(4, 4096, 4096)["kernel_name"] == "stream"   # BF16 weights when forced
        with pytest.raises(rg.RgError):
            rg.rg_plan(1, 4096, 4100)               # BF16: K % 8 == 0 only
        with pytest.raises(rg.RgError):
            rg.rg_plan_f32w(5, 4096, 4096)          # M <= 4 only
        rg.rg_linear_set_launch(kernel="ktile")
        assert rg.rg_plan_f32w(1, 4096, 4096)["kernel_name"] == "ktile"
    finally:
        rg.rg_linear_set_launch(None)
    L = rg.lib
    assert L.rg_linear_f32w(None, 0x1000, 0x2000, 1, 1, 1, None) == rg.RG_ERR_INVAL
    assert L.rg_linear_f32w(0x1000, 0x2002, 0x3000, 1, 1, 1, None) == rg.RG_ERR_ALIGN
    assert L.rg_linear_f32w(0x1000, 0x2000, 0x1000, 1, 1, 1, None) == rg.RG_ERR_ALIAS
    assert L.rg_linear_f32w(0x1000, 0x2000, 0x3000, 1, 0, 1, None) == rg.RG_ERR_INVAL


def test_attention_header_exports_and_host_checks():
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "rg_attn.h")).read(), flags=re.S)
    names = sorted(set(re.findall(r"^\s*(?:int|int64_t)\s+(rg_\w+)\s*\(", text, flags=re.M)))
    assert sorted(rg.ATTN_EXPORTS) == names
    lib = ctypes.CDLL(rg.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    ws = rg.rg_attn_workspace_size(16, 32, 4096, 128)
    assert ws >= 4 * (16 * 32 * 4096 + 2 * 16 * 32 * 16 + 16 * 32 * 16 * 128)
    assert rg.rg_attn_workspace_size(0, 32, 4096, 128) == 0
    L = rg.lib
    a = 0x100000
    # null, bad group, bad D, small workspace, misalignment -- all before any device call
    assert L.rg_attn_decode(None, a, a, a, a, 1, 1, 1, 16, 64, 1.0, a, 1 << 20, None) == rg.RG_ERR_INVAL
    assert L.rg_attn_decode(a, a, a, a, a, 1, 3, 2, 16, 64, 1.0, a, 1 << 20, None) == rg.RG_ERR_INVAL
    assert L.rg_attn_decode(a, a, a, a, a, 1, 9, 1, 16, 64, 1.0, a, 1 << 20, None) == rg.RG_ERR_INVAL
    assert L.rg_attn_decode(a, a, a, a, a, 1, 1, 1, 16, 60, 1.0, a, 1 << 20, None) == rg.RG_ERR_INVAL
    assert L.rg_attn_decode(a, a, a, a, a, 1, 1, 1, 16, 264, 1.0, a, 1 << 20, None) == rg.RG_ERR_INVAL
    assert L.rg_attn_decode(a, a, a, a, a, 1, 1, 1, 16, 64, 1.0, a, 8, None) == rg.RG_ERR_INVAL
    assert L.rg_attn_decode(a + 4, a, a, a, 0x900000, 1, 1, 1, 16, 64, 1.0, 0xA00000, 1 << 20, None) == rg.RG_ERR_ALIGN
    assert L.rg_attn_decode(0x100000, 0x200000, 0x300000, 0x400000, 0x100000, 1, 1, 1, 16, 64, 1.0, 0xA00000,
                            1 << 20, None) == rg.RG_ERR_ALIAS


def test_attention_kernels_use_only_ieee_operations():
    src = os.path.join(ROOT, "paper_2609_25624_amd", "csrc", "rg_attn.hip")
    code = re.sub(r"//.*", "", open(src).read())
    for bad in ("atomic", "mfma", "__expf", "__builtin_expf", "exp2f", "fast-math"):
        assert bad not in code, bad
    asm = _device_asm("rg_attn.hip")
    insts = set(re.findall(r"^\s+(v_[a-z0-9_]+)", asm, flags=re.M))
    for i in insts:
        assert not re.match(r"v_(mfma|dot\d|pk_(fma|mul|add)_f32|mad_f32|mac_f32|exp_f32|log_f32|fma_mix|mad_mix)", i), i
    assert "v_div_fixup_f32" in insts          # the correctly rounded division
    modes = re.findall(r"\.amdhsa_float_denorm_mode_32\s+(\d+)", asm)
    assert modes and set(modes) == {"3"}


def test_attention_noalloc_host_checks():
    """The no-allocation attention entry point refuses a workspace beyond its static scratch, and
    bad arguments, before any device call (so these run without a GPU)."""
    L = rg.lib
    assert rg.ATTN_SCRATCH_BYTES == 64 << 20
    q, out, lens, kc, vc = 0x1000000, 0x2000000, 0x3000000, 0x10000000, 0x20000000
    B, H, Hkv, Lmax, D = 1, 8, 1, 2_200_000, 8
    assert rg.rg_attn_workspace_size(B, H, Lmax, D) > rg.ATTN_SCRATCH_BYTES
    assert L.rg_attn_decode_noalloc(q, kc, vc, lens, out, B, H, Hkv, Lmax, D, 1.0, None) == rg.RG_ERR_RANGE
    assert rg.rg_attn_workspace_size(B, H, 2_000_000, D) < rg.ATTN_SCRATCH_BYTES   # the limit is the size
    assert L.rg_attn_decode_noalloc(None, kc, vc, lens, out, 1, 1, 1, 16, 64, 1.0, None) == rg.RG_ERR_INVAL
    assert L.rg_attn_decode_noalloc(q, kc, vc, lens, out, 1, 3, 2, 16, 64, 1.0, None) == rg.RG_ERR_INVAL
    assert L.rg_attn_decode_noalloc(q + 4, kc, vc, lens, out, 1, 1, 1, 16, 64, 1.0, None) == rg.RG_ERR_ALIGN
    assert L.rg_attn_decode_noalloc(q, kc, vc, lens, q, 1, 1, 1, 16, 64, 1.0, None) == rg.RG_ERR_ALIAS


def test_noalloc_scratch_is_a_static_device_array_taken_by_symbol_address():
    """The scratch lives in a file-scope __device__ array whose address host code takes with
    hipGetSymbolAddress; the array's name never reaches a kernel argument."""
    src = open(os.path.join(ROOT, "paper_2609_25624_amd", "csrc", "rg_api.cpp")).read()
    code = re.sub(r"//.*", "", src)
    assert re.search(r"^__device__ __align__\(256\) uint8_t scratch\[RG_ATTN_SCRATCH_BYTES\];", code, re.M)
    assert code.count("HIP_SYMBOL(scratch)") == 1
    uses = [m.start() for m in re.finditer(r"\bscratch\b", code)]
    assert len(uses) == 2, "the array is named only in its definition and in hipGetSymbolAddress"
    body = code[code.index("int rg_attn_decode_noalloc("):]
    body = body[:body.index("\n}\n")]
    for bad in ("hipMalloc", "hipFree", "hipMemset", "hipHostMalloc", "new ", "malloc("):
        assert bad not in body, bad


def test_baseline_library_exports_and_host_checks():
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "rg_baseline.h")).read(), flags=re.S)
    names = sorted(set(re.findall(r"^\s*int\s+(rg_\w+)\s*\(", text, flags=re.M)))
    from paper_2609_25624_amd import baseline
    assert sorted(baseline.EXPORTS) == names
    L = baseline.lib
    a, b, c, d = 0x1000000, 0x2000000, 0x3000000, 0x4000000
    assert L.rg_linear_cast_baseline(None, b, c, d, 1, 1, 1, None) == rg.RG_ERR_INVAL
    assert L.rg_linear_cast_baseline(a, b, c, d, 1, 0, 1, None) == rg.RG_ERR_INVAL
    assert L.rg_linear_cast_baseline(a, b, c, d, 1, 1 << 31, 1, None) == rg.RG_ERR_INVAL
    assert L.rg_linear_cast_baseline(a + 2, b, c, d, 1, 1, 1, None) == rg.RG_ERR_ALIGN
    assert L.rg_linear_cast_baseline(a, b, a, d, 1, 1, 1, None) == rg.RG_ERR_ALIAS       # w_tmp over x
    assert L.rg_linear_cast_baseline(a, b, c, c, 1, 1, 1, None) == rg.RG_ERR_ALIAS       # y over w_tmp


def test_inline_assembly_writes_no_register_asynchronously():
    """A vector or scalar memory load issued from inline assembly writes its destination registers
    when the data returns, which the compiler cannot see: it may copy or reuse those registers
    before then (a build that loaded x this way reused a pending destination for a load address,
    and faulted).  The only memory instruction the library's inline assembly may issue is the
    global->LDS DMA (no register destination); every other asm instruction is synchronous."""
    allowed = {"s_nop", "s_mov_b32", "s_add_u32", "global_load_lds_dwordx4", "s_waitcnt", "v_fmac_f32_dpp"}
    for f in ("rg_kernels.hip", "rg_wtile.hip", "rg_attn.hip"):
        asm = _device_asm(f)
        blocks = re.findall(r";;#ASMSTART\n(.*?);;#ASMEND", asm, flags=re.S)
        ops = {ln.split()[0] for blk in blocks for ln in blk.splitlines() if ln.strip() and not ln.strip().startswith(";")}
        assert ops <= allowed, (f, sorted(ops - allowed))


def test_inline_lds_dma_never_reads_m0_right_after_writing_it():
    """On this generation an LDS DMA needs one wait state after a scalar write of M0 (its LDS
    address); the compiler inserts it for DMA it emits itself, not inside inline assembly.
    Every global_load_lds in the library's inline assembly follows an instruction that is not
    an M0 write."""
    n = 0
    for f in ("rg_kernels.hip", "rg_attn.hip"):
        for blk in re.findall(r";;#ASMSTART\n(.*?);;#ASMEND", _device_asm(f), flags=re.S):
            lines = [ln.strip() for ln in blk.splitlines() if ln.strip() and not ln.strip().startswith(";")]
            for i, ln in enumerate(lines):
                if ln.startswith("global_load_lds"):
                    n += 1
                    assert i > 0 and not re.match(r"s_\w+\s+m0,", lines[i - 1]), (f, lines[max(0, i - 2):i + 1])
    assert n > 0


def test_probe_library_exports_and_host_checks():
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "rg_probe.h")).read(), flags=re.S)
    names = sorted(set(re.findall(r"^\s*int\s+(rg_\w+)\s*\(", text, flags=re.M)))
    from paper_2609_25624_amd import probe
    assert sorted(probe.EXPORTS) == names
    L = probe.lib
    assert L.rg_probe_read(None, 8192, 0x1000, 1, None) == 1
    assert L.rg_probe_read(0x1000, 8000, 0x2000, 1, None) == 1          # not a multiple of 8 KB
    assert L.rg_probe_read(0x1008, 8192, 0x2000, 1, None) == 1          # misaligned
    assert L.rg_probe_read(0x1000, 8192, 0x2000, 0, None) == 1          # no workgroups
    assert L.rg_probe_fma(0, 8, None, 1, 1, None) == 1
    assert L.rg_probe_fma(5, 8, 0x1000, 1, 1, None) == 1                # no such mode
    assert L.rg_probe_fma(0, 12, 0x1000, 1, 1, None) == 1               # 8 or 16 chains
    assert L.rg_probe_fma(0, 8, 0x1000, 0, 1, None) == 1
    assert L.rg_probe_fma(0, 8, 0x1000, 1, 0, None) == 1
