"""The C-ABI library (CPU only): it loads, exports every function include/fp4root.h
declares, and validates arguments on the host before any GPU work."""
import ctypes
import os
import re

import pytest

from paper_2607_04422_amd import fp4root as F

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib():
    if not os.path.exists(F.LIB_PATH):
        pytest.fail("libfp4root.so is not built (run __graft_entry__.build())")
    return F.load()


def test_exports_every_declared_symbol():
    lib = _lib()
    declared = F.header_symbols()
    assert len(declared) >= 13
    for name in declared:
        assert hasattr(lib, name), f"{name} declared in include/fp4root.h but not exported"
    # and nothing else public: every exported fp4root_* function is declared
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", F.LIB_PATH], capture_output=True, text=True).stdout
    exported = sorted(set(re.findall(r" T (fp4root_\w+)", out)))
    assert exported == declared


def test_host_helpers():
    _lib()
    assert F.fp4root_version() == 200
    assert F.status_string(-3).startswith("workspace")
    co = F.fp4root_default_coeffs(3072, 8192, 5)
    assert len(co) == 5 and all(len(r) == 3 for r in co)
    # the table is keyed by aspect ratio only
    assert F.fp4root_default_coeffs(8192, 3072, 5) == co
    assert F.fp4root_default_coeffs(1024, 3072, 5) == co


def test_workspace_queries():
    lib = _lib()
    assert lib.fp4root_quantize_workspace(1, 64, 64, 0) >= 256
    assert lib.fp4root_quantize_workspace(4, 64, 64, 1) > lib.fp4root_quantize_workspace(4, 64, 64, 0)
    a = lib.fp4root_ns_step_workspace(2, 256, 512, 6)
    assert a >= 2 * (256 * 512 + 256 * 256 * 4)
    assert lib.fp4root_ns_step_workspace(2, 250, 512, 6) == 0
    mats = (F.Matrix * 2)(F.Matrix(16, 16, 256, 512, 512, 512), F.Matrix(32, 32, 512, 256, 256, 256))
    cfg = F.NsConfig(5, None, 7, 0.99, 1e-7, 0)
    assert lib.fp4root_orthogonalize_workspace(mats, 2, ctypes.byref(cfg)) > 0
    bad = F.NsConfig(5, None, 7 | 64, 0.99, 1e-7, 0)
    assert lib.fp4root_orthogonalize_workspace(mats, 2, ctypes.byref(bad)) == 0
    # binary32 accumulation is an NVFP4-path option: accepted alone, rejected with the BF16 path
    fp32 = F.NsConfig(5, None, 7 | F.F_FP32_ACCUM, 0.99, 1e-7, 0)
    assert lib.fp4root_orthogonalize_workspace(mats, 2, ctypes.byref(fp32)) == \
        lib.fp4root_orthogonalize_workspace(mats, 2, ctypes.byref(cfg))
    both = F.NsConfig(5, None, F.F_CLIP | F.F_BF16_PATH | F.F_FP32_ACCUM, 0.99, 1e-7, 0)
    assert lib.fp4root_orthogonalize_workspace(mats, 2, ctypes.byref(both)) == 0


def test_product_tiling_switch():
    """Host-side setting: returns the previous mode, rejects modes outside 0..2."""
    lib = _lib()
    assert lib.fp4root_set_product_tiling(1) == 0
    assert lib.fp4root_set_product_tiling(2) == 1
    assert lib.fp4root_set_product_tiling(3) == -1
    assert lib.fp4root_set_product_tiling(-1) == -1
    assert lib.fp4root_set_product_tiling(0) == 2


def test_argument_errors_are_synchronous():
    lib = _lib()
    vp = ctypes.c_void_p
    fake = vp(0x100000)   # never dereferenced: validation fails before any launch
    ws = vp(0x200000)
    # null input
    assert lib.fp4root_quantize(None, 1, 64, 64, 64, 4096, 1, 0, 0.99, 0, 0, fake, fake, fake, None,
                                ws, 1 << 20, None) == -1
    # shape not a multiple of 16
    assert lib.fp4root_quantize(fake, 1, 60, 64, 64, 4096, 1, 0, 0.99, 0, 0, fake, fake, fake, None,
                                ws, 1 << 20, None) == -2
    # bad axis, bad flag, bad quantile
    assert lib.fp4root_quantize(fake, 1, 64, 64, 64, 4096, 2, 0, 0.99, 0, 0, fake, fake, fake, None,
                                ws, 1 << 20, None) == -1
    assert lib.fp4root_quantize(fake, 1, 64, 64, 64, 4096, 1, 8, 0.99, 0, 0, fake, fake, fake, None,
                                ws, 1 << 20, None) == -1
    assert lib.fp4root_quantize(fake, 1, 64, 64, 64, 4096, 1, 1, 1.5, 0, 0, fake, fake, fake, None,
                                ws, 1 << 20, None) == -1
    # workspace too small
    assert lib.fp4root_quantize(fake, 1, 64, 64, 64, 4096, 1, 0, 0.99, 0, 0, fake, fake, fake, None,
                                ws, 8, None) == -3
    # ns_step: non-finite coefficient, bad shape, workspace
    nan = float("nan")
    assert lib.fp4root_ns_step(fake, 1, 64, 64, 4096, nan, 0.0, 0.0, 6, 0, 0, None, ws, 1 << 30, None) == -1
    assert lib.fp4root_ns_step(fake, 1, 64, 72, 4608, 1.0, 0.0, 0.0, 6, 0, 0, None, ws, 1 << 30, None) == -2
    assert lib.fp4root_ns_step(fake, 1, 64, 64, 4096, 1.0, 0.0, 0.0, 6, 0, 0, None, ws, 16, None) == -3
    # a side above 2^21 (products address 128-row tiles with 32-bit byte offsets)
    big = (1 << 21) + 16
    assert lib.fp4root_ns_step(fake, 1, 64, big, 64 * big, 1.0, 0.0, 0.0, 6, 0, 0, None, ws, 1 << 30,
                               None) == -2
    assert lib.fp4root_quantize(fake, 1, 64, big, big, 64 * big, 1, 0, 0.99, 0, 0, fake, fake, fake, None,
                                ws, 1 << 40, None) == -2
    # orthogonalize: unaligned pointer, in-place with different ld, bad count
    cfg = F.NsConfig(5, None, 7, 0.99, 1e-7, 0)
    m1 = (F.Matrix * 1)(F.Matrix(0x100004, 0x300000, 64, 64, 64, 64))
    assert lib.fp4root_orthogonalize(m1, 1, ctypes.byref(cfg), ws, 1 << 30, None) == -1
    m2 = (F.Matrix * 1)(F.Matrix(0x100000, 0x100000, 64, 64, 64, 128))
    assert lib.fp4root_orthogonalize(m2, 1, ctypes.byref(cfg), ws, 1 << 30, None) == -1
    m3 = (F.Matrix * 1)(F.Matrix(0x100000, 0x300000, 64, 40, 64, 40))
    assert lib.fp4root_orthogonalize(m3, 1, ctypes.byref(cfg), ws, 1 << 30, None) == -2
    assert lib.fp4root_orthogonalize(m3, -1, ctypes.byref(cfg), ws, 1 << 30, None) == -1
    assert lib.fp4root_orthogonalize(m1, 1, None, ws, 1 << 30, None) == -1


def test_binding_refuses_cpu_tensors():
    import torch
    _lib()
    with pytest.raises(TypeError):
        F.fp4root_quantize(torch.zeros(16, 16))
    with pytest.raises(TypeError):
        F.fp4root_ns_step(torch.zeros(16, 16), 1.0, 0.0, 0.0)


def test_root_step_and_qadamw_reject_before_any_launch():
    # every parameter is checked before the first launch: a bad second parameter
    # fails the call synchronously (the fake pointers are never dereferenced)
    lib = _lib()
    ws = ctypes.c_void_p(0x200000)
    good = F.Param(0x100000, 0x110000, 0x120000, 0x130000, 0x140000, 0x150000, 64, 128, 0.0)
    cfg = F.RootConfig(0.01, 0.1, 0.9, 6, 0, 0)
    ns_cfg = F.NsConfig(5, None, 7, 0.99, 1e-7, 0)
    for field, value, want in (("m_codes", 0, -1), ("m_codes", 0x130001, -1), ("g", 0x110004, -1),
                               ("scale", -1.0, -1), ("rows", 72, -2)):
        bad = F.Param(*[getattr(good, f) for f, _ in F.Param._fields_])
        setattr(bad, field, value)
        params = (F.Param * 2)(good, bad)
        assert lib.fp4root_root_step(params, 2, ctypes.byref(cfg), ctypes.byref(ns_cfg), ws, 1 << 40,
                                     None) == want, field
    # quantized-state AdamW: the first-moment output may not overlap the gradient at all
    n = 4096
    g = 0x100000
    for m in (g, g + 64, g - 64):
        assert lib.fp4root_qadamw_update(0x300000, g, m, n, 0x400000, 0x410000, 0x420000, 0x430000, 0x440000,
                                         0x450000, 1e-3, 0.1, 0.9, 0.95, 1e-8, 6, 0, 0, ws, 1 << 30, None) == -1
