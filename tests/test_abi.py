"""C ABI: the library loads, exports every declared symbol, and rejects bad
arguments on the host before touching the GPU (CPU only: no kernel runs)."""

import ctypes
import os
import re

import pytest

from paper_2606_25040_amd import ops

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "chorus.h")

FAKE = 0x10000           # aligned, never dereferenced: every call below fails validation first


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ops.LIB_PATH):
        pytest.fail("libchorus.so is not built (run __graft_entry__.build())")
    return ops.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(chorus_\w+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 14
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(ops.EXPORTS) == names


def test_status_strings_and_version(lib):
    assert lib.chorus_status_string(0) == b"CHORUS_OK"
    assert lib.chorus_status_string(3) == b"CHORUS_ERR_CAPACITY"
    assert lib.chorus_version() >= 100


def t4(B=1, S=100, H=2):
    return ops.Tensor(FAKE, S * H * 128, H * 128, 128)


def shape(B=1, S=100, H=2, D=128):
    return ops.Shape(B, S, H, D)


def build(lib, shp, q=None, top_p=0.5, mk=0.1, cap=None, ws_bytes=None, dtype=ops.BF16, ks=None, kvb=64):
    n = (shp.S + 63) // 64
    rows = shp.B * shp.H * n
    cap = rows * n if cap is None else cap
    need = lib.chorus_build_block_mask_workspace_size(ctypes.byref(shp))
    ws = need if ws_bytes is None else ws_bytes
    qq = q or t4(shp.B, shp.S, shp.H)
    return lib.chorus_build_block_mask(dtype, ctypes.byref(shp), ctypes.byref(qq), ctypes.byref(qq),
                                       0.088, top_p, mk, kvb, ks, FAKE, FAKE, cap, None, FAKE, ws, None)


def test_builder_argument_checks(lib):
    assert build(lib, shape(D=64)) == 2
    assert build(lib, shape(S=0)) == 1
    assert build(lib, shape(), top_p=1.5) == 1
    assert build(lib, shape(), top_p=float("nan")) == 1
    assert build(lib, shape(), mk=-0.1) == 1
    assert build(lib, shape(), cap=3) == 3
    assert build(lib, shape(), ws_bytes=16) == 5
    assert build(lib, shape(), dtype=ops.FP8_E4M3) == 2
    assert build(lib, shape(S=64 * 4097)) == 2
    bad = ops.Tensor(FAKE + 8, 100 * 2 * 128, 2 * 128, 128)
    assert build(lib, shape(), q=bad) == 1
    bad = ops.Tensor(FAKE, 100 * 2 * 128, 2 * 128 + 4, 128)
    assert build(lib, shape(), q=bad) == 1
    assert b"stride" in lib.chorus_last_error()


def build_noalloc(lib, shp, top_p=0.5, mk=0.1, cap=None, dtype=ops.BF16, kvb=64):
    n = (shp.S + 63) // 64
    nk = (shp.S + kvb - 1) // kvb
    rows = shp.B * shp.H * n
    cap = rows * nk if cap is None else cap
    qq = t4(shp.B, shp.S, shp.H)
    return lib.chorus_build_block_mask_noalloc(dtype, ctypes.byref(shp), ctypes.byref(qq), ctypes.byref(qq),
                                               0.088, top_p, mk, kvb, None, FAKE, FAKE, cap, None, None)


def test_noalloc_builder_rejects_before_any_device_call(lib):
    """Every rejection happens in the host checks, before the first device
    call; in particular a shape whose single head does not fit the fixed
    scratch (n_blocks = 4096: 8.4 MB of pooled means plus 134 MB of scores)
    is CHORUS_ERR_CAPACITY, and fp8 input is not taken."""
    assert build_noalloc(lib, shape(S=64 * 4096, H=1)) == 3
    assert b"scratch" in lib.chorus_last_error()
    assert build_noalloc(lib, shape(S=64 * 2800, H=1)) == 3
    assert build_noalloc(lib, shape(), dtype=ops.FP8_E4M3) == 2
    assert build_noalloc(lib, shape(D=64)) == 2
    assert build_noalloc(lib, shape(), top_p=1.5) == 1
    assert build_noalloc(lib, shape(), cap=3) == 3
    assert build_noalloc(lib, shape(), kvb=96) == 2


def attn(lib, shp, mask, dtype=ops.BF16, scales=(None, None, None), sched=None, sm=0.088, ks=None):
    t = t4(shp.B, shp.S, shp.H)
    return lib.chorus_block_sparse_attn_fwd(dtype, ctypes.byref(shp), ctypes.byref(t), ctypes.byref(t),
                                            ctypes.byref(t), *scales, ctypes.byref(mask),
                                            sched, sm, ks, ctypes.byref(t), None, None, 0, None)


def test_attention_argument_checks(lib):
    shp = shape(B=2, S=100, H=2)
    ok = ops.Mask(1, 2, 2, 64, FAKE, FAKE)
    assert attn(lib, shp, ops.Mask(1, 2, 2, 256, FAKE, FAKE)) == 2     # kv block 256
    assert attn(lib, shp, ops.Mask(1, 2, 2, 32, FAKE, FAKE)) == 2      # kv block 32
    assert attn(lib, shp, ops.Mask(3, 2, 2, 64, FAKE, FAKE)) == 1      # mask_batch
    assert attn(lib, shp, ops.Mask(1, 3, 2, 64, FAKE, FAKE)) == 1      # H
    assert attn(lib, shp, ops.Mask(1, 2, 3, 64, FAKE, FAKE)) == 1      # n_blocks
    assert attn(lib, shp, ops.Mask(1, 2, 2, 64, None, FAKE)) == 1      # null row_ptr
    assert attn(lib, shp, ok, dtype=ops.FP8_E4M3) == 1                 # fp8 without scales
    assert attn(lib, shp, ok, scales=(FAKE, FAKE, FAKE)) == 1          # scales on bf16
    assert attn(lib, shp, ok, dtype=7) == 2
    assert attn(lib, shp, ok, sm=0.0) == 1
    sched = ops.Schedule(FAKE, 5)
    assert attn(lib, shp, ok, sched=ctypes.byref(sched)) == 1
    assert attn(lib, shape(D=64), ok) == 2


def test_other_entry_points_check_arguments(lib):
    shp = shape()
    t = t4()
    assert lib.chorus_quantize_fp8_blockwise(ops.FP8_E4M3, ctypes.byref(shp), ctypes.byref(t),
                                             ctypes.byref(t), FAKE, None) == 2
    assert lib.chorus_quantize_fp8_blockwise(ops.BF16, ctypes.byref(shp), ctypes.byref(t),
                                             ctypes.byref(t), None, None) == 1
    m = ops.Mask(1, 2, 2, 64, FAKE, FAKE)
    assert lib.chorus_plan_block_mask(ctypes.byref(shp), ctypes.byref(m), None, None, 0, None) == 1
    assert lib.chorus_validate_block_mask(ctypes.byref(m), 10, None, None) == 1
    assert lib.chorus_build_block_mask_workspace_size(ctypes.byref(shape(S=75600, H=40))) > 0


def test_block_sums_entry_points_check_arguments(lib):
    """The quantiser with block sums and the builder from sums reject bad
    arguments on the host, before any device work."""
    shp = shape()
    t = t4()
    ks_bad = ops.KeyScale(101, 1.5)                  # n_first > S
    q = lib.chorus_quantize_fp8_blockwise_sums
    assert q(ops.FP8_E4M3, ctypes.byref(shp), ctypes.byref(t), ctypes.byref(t), FAKE, None, FAKE, None) == 2
    assert q(ops.BF16, ctypes.byref(shp), ctypes.byref(t), ctypes.byref(t), FAKE, None, None, None) == 1
    assert q(ops.BF16, ctypes.byref(shp), ctypes.byref(t), ctypes.byref(t), None, None, FAKE, None) == 1
    assert q(ops.BF16, ctypes.byref(shp), ctypes.byref(t), ctypes.byref(t), FAKE, None, FAKE + 4, None) == 1
    assert q(ops.BF16, ctypes.byref(shp), ctypes.byref(t), ctypes.byref(t), FAKE, ctypes.byref(ks_bad), FAKE,
             None) == 1
    assert q(ops.BF16, ctypes.byref(shape(D=64)), ctypes.byref(t), ctypes.byref(t), FAKE, None, FAKE, None) == 2
    b = lib.chorus_build_block_mask_from_sums
    n = 2
    need = lib.chorus_build_block_mask_workspace_size(ctypes.byref(shp))
    cap = 2 * n * n

    def call(qs=FAKE, kss=FAKE, top_p=0.5, mk=0.1, kvb=64, rp=FAKE, ci=FAKE, c=cap, ws=FAKE, wsb=need, sm=0.088):
        return b(ctypes.byref(shp), qs, kss, sm, top_p, mk, kvb, rp, ci, c, None, ws, wsb, None)

    assert call(qs=None) == 1
    assert call(kss=None) == 1
    assert call(qs=FAKE + 4) == 1
    assert call(top_p=1.5) == 1
    assert call(mk=-0.1) == 1
    assert call(kvb=96) == 2
    assert call(rp=None) == 1
    assert call(c=cap - 1) == 3
    assert call(sm=float("inf")) == 1
    assert call(wsb=need - 1) == 5


def test_block_sums_binding_checks_shapes_on_the_host(lib):
    """The Python binding of the builder from block sums rejects mismatched
    or mis-sized sums before any device call (CPU tensors suffice)."""
    import torch
    qs = torch.zeros((1, 2, 16, 128), dtype=torch.float64)
    with pytest.raises(ValueError):
        ops.build_block_mask_from_sums(qs, torch.zeros((1, 2, 15, 128), dtype=torch.float64), 1000, 0.5, 0.1)
    with pytest.raises(ValueError):
        ops.build_block_mask_from_sums(qs, qs.float(), 1000, 0.5, 0.1)
    with pytest.raises(ValueError):   # S = 1000 has 16 blocks of 64 tokens, not 15
        short = torch.zeros((1, 2, 15, 128), dtype=torch.float64)
        ops.build_block_mask_from_sums(short, short, 1000, 0.5, 0.1)
    with pytest.raises(ValueError):
        ops.quantize_fp8_blockwise_sums(torch.zeros((1, 100, 2, 128), dtype=torch.bfloat16),
                                        block_sums=torch.zeros((1, 2, 1, 128), dtype=torch.float64))


def test_block_mass_selection_and_coverage_check_arguments(lib):
    shp = shape(B=1, S=100, H=2)
    t = t4()
    assert lib.chorus_attn_block_mass(ops.FP8_E4M3, ctypes.byref(shp), ctypes.byref(t), ctypes.byref(t),
                                      FAKE, 0.088, 64, None, FAKE, None) == 2
    assert lib.chorus_attn_block_mass(ops.BF16, ctypes.byref(shp), ctypes.byref(t), ctypes.byref(t),
                                      None, 0.088, 64, None, FAKE, None) == 1
    assert lib.chorus_attn_block_mass(ops.BF16, ctypes.byref(shp), ctypes.byref(t), ctypes.byref(t),
                                      FAKE, -1.0, 64, None, FAKE, None) == 1
    assert lib.chorus_attn_block_mass(ops.BF16, ctypes.byref(shape(D=64)), ctypes.byref(t), ctypes.byref(t),
                                      FAKE, 0.088, 64, None, FAKE, None) == 2
    need = lib.chorus_select_block_mask_workspace_size(ctypes.byref(shp))
    assert need > 0
    sel = lib.chorus_select_block_mask
    assert sel(ctypes.byref(shp), FAKE, 64, 1.5, 0.0, FAKE, FAKE, 8, FAKE, need, None) == 1
    assert sel(ctypes.byref(shp), FAKE, 64, 0.5, 0.0, FAKE, FAKE, 7, FAKE, need, None) == 3
    assert sel(ctypes.byref(shp), FAKE, 64, 0.5, 0.0, FAKE, FAKE, 8, FAKE, 16, None) == 5
    assert sel(ctypes.byref(shp), None, 64, 0.5, 0.0, FAKE, FAKE, 8, FAKE, need, None) == 1
    assert sel(ctypes.byref(shape(S=64 * 4097)), FAKE, 64, 0.5, 0.0, FAKE, FAKE, 1 << 40, FAKE, 1 << 40,
               None) == 2
    m = ops.Mask(1, 2, 2, 64, FAKE, FAKE)
    assert lib.chorus_mask_coverage(ctypes.byref(shp), ctypes.byref(m), None, FAKE, None) == 1
    assert lib.chorus_mask_coverage(ctypes.byref(shp), ctypes.byref(ops.Mask(1, 3, 2, 64, FAKE, FAKE)),
                                    FAKE, FAKE, None) == 1



def test_visit_refresh_checks_arguments(lib):
    vb = lambda *a: lib.chorus_visit_map_bytes(ctypes.byref(ops.Mask(*a, None, None)))
    assert vb(1, 40, 1182, 64) == 40 * 1182 * 37 * 4
    assert vb(1, 40, 1182, 128) == 40 * 1182 * 19 * 4          # 591 kv blocks per row
    assert vb(0, 40, 1182, 64) == 0
    assert vb(1, 40, 1182, 96) == 0
    assert lib.chorus_visit_map_bytes(None) == 0
    m = ops.Mask(1, 2, 10, 64, FAKE, FAKE)
    assert lib.chorus_visit_refresh_workspace_size(ctypes.byref(m)) >= 20 * 4 + 20 * 4
    assert lib.chorus_visit_reset(None, FAKE, None) == 1
    assert lib.chorus_visit_update(ctypes.byref(m), None, None) == 1
    assert lib.chorus_visit_update(ctypes.byref(ops.Mask(1, 2, 10, 256, FAKE, FAKE)), FAKE, None) == 2
    assert lib.chorus_visit_update(ctypes.byref(ops.Mask(1, 2, 4097, 64, FAKE, FAKE)), FAKE, None) == 2
    assert lib.chorus_visit_update(ctypes.byref(ops.Mask(1, 2, 10, 64, None, FAKE)), FAKE, None) == 1
    need = lib.chorus_visit_refresh_workspace_size(ctypes.byref(m))
    assert lib.chorus_visit_refresh(ctypes.byref(m), FAKE, FAKE, FAKE, 2 * 10 * 10 - 1, FAKE, need, None) == 3
    assert lib.chorus_visit_refresh(ctypes.byref(m), FAKE, FAKE, FAKE, 2 * 10 * 10, FAKE, need - 4, None) == 5
    assert lib.chorus_visit_refresh(ctypes.byref(m), None, FAKE, FAKE, 2 * 10 * 10, FAKE, need, None) == 1


def test_key_scale_checks(lib):
    shp = shape(B=2, S=100, H=2)
    ok = ops.Mask(1, 2, 2, 64, FAKE, FAKE)
    bad_n = ctypes.byref(ops.KeyScale(101, 2.0))
    neg_n = ctypes.byref(ops.KeyScale(-1, 2.0))
    nan_b = ctypes.byref(ops.KeyScale(10, float("nan")))
    inf_b = ctypes.byref(ops.KeyScale(10, float("inf")))
    for ks in (bad_n, neg_n, nan_b, inf_b):
        assert attn(lib, shp, ok, ks=ks) == 1
        assert build(lib, shape(), ks=ks) == 1
        t = t4()
        assert lib.chorus_attn_block_mass(ops.BF16, ctypes.byref(shape(B=1, S=100, H=2)), ctypes.byref(t),
                                          ctypes.byref(t), FAKE, 0.088, 64, ks, FAKE, None) == 1
    assert b"key_scale" in lib.chorus_last_error()


def test_fp8_builder_checks_arguments(lib):
    shp = shape()
    n = (shp.S + 63) // 64
    cap = shp.B * shp.H * n * n
    need = lib.chorus_build_block_mask_workspace_size(ctypes.byref(shp))
    t8 = ops.Tensor(FAKE, 100 * 2 * 128, 2 * 128, 128)
    f = lib.chorus_build_block_mask_fp8
    assert f(ctypes.byref(shp), ctypes.byref(t8), None, ctypes.byref(t8), FAKE, 0.088, 0.5, 0.1, 64, None,
             FAKE, FAKE, cap, None, FAKE, need, None) == 1
    assert f(ctypes.byref(shp), ctypes.byref(t8), FAKE, ctypes.byref(t8), FAKE, 0.088, 0.5, 0.1, 64, None,
             FAKE, FAKE, cap - 1, None, FAKE, need, None) == 3
    assert f(ctypes.byref(shape(D=64)), ctypes.byref(t8), FAKE, ctypes.byref(t8), FAKE, 0.088, 0.5, 0.1, 64, None,
             FAKE, FAKE, cap, None, FAKE, need, None) == 2
    assert f(ctypes.byref(shp), ctypes.byref(ops.Tensor(FAKE + 4, 100 * 2 * 128, 2 * 128, 128)), FAKE,
             ctypes.byref(t8), FAKE, 0.088, 0.5, 0.1, 64, None, FAKE, FAKE, cap, None, FAKE, need, None) == 1


def test_kv_block_checks(lib):
    assert build(lib, shape(), kvb=96) == 2
    assert build(lib, shape(), kvb=128) != 2 or b"kv_block" not in lib.chorus_last_error()
    # kv blocks of 128: the worst-case capacity is rows * ceil(S / 128)
    shp = shape(S=300)
    rows = 1 * 2 * 5
    assert build(lib, shp, kvb=128, cap=rows * 3 - 1) == 3
    t = t4()
    assert lib.chorus_attn_block_mass(ops.BF16, ctypes.byref(shape(B=1, S=100, H=2)), ctypes.byref(t),
                                      ctypes.byref(t), FAKE, 0.088, 100, None, FAKE, None) == 2
    need = lib.chorus_select_block_mask_workspace_size(ctypes.byref(shp))
    assert lib.chorus_select_block_mask(ctypes.byref(shp), FAKE, 128, 0.5, 0.0, FAKE, FAKE, rows * 3 - 1,
                                        FAKE, need, None) == 3
    assert lib.chorus_validate_block_mask(ctypes.byref(ops.Mask(1, 2, 5, 100, FAKE, FAKE)), 10, FAKE, None) == 2


def test_header_is_plain_c_and_a_c_caller_links(tmp_path):
    """Compile a C99 caller against include/chorus.h with gcc and run it:
    host-side calls only (argument validation, sizes, strings)."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    exe = tmp_path / "abi_c_caller"
    lib_dir = os.path.dirname(ops.LIB_PATH)
    cmd = [gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "abi_c_caller.c"), "-L", lib_dir, "-lchorus",
           f"-Wl,-rpath,{lib_dir}", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr
