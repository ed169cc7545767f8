"""C-ABI contract tests that need no GPU: the library loads, exports every
symbol include/shiftquant.h declares, and rejects bad arguments synchronously
(before any HIP call) with the documented status codes."""
import ctypes as ct
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "shiftquant.h")


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:sq_status|const char\*)\s+(sq_\w+)\s*\(", src, re.M)))


@pytest.fixture(scope="module")
def sq():
    from paper_2411_10948_amd import shiftquant
    if not os.path.exists(shiftquant.LIB_PATH):
        from paper_2411_10948_amd import build
        build.build()
    return shiftquant


def test_header_declares_the_five_calls():
    names = _declared()
    for n in ["sq_quantize_grad", "sq_quantize_tensor", "sq_gemm_dgrad", "sq_gemm_wgrad", "sq_dequant"]:
        assert n in names


def test_library_exports_every_declared_symbol(sq):
    names = _declared()
    out = subprocess.run(["nm", "-D", "--defined-only", sq.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(l.split()[-1] for l in out.splitlines() if " T " in l)
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    assert sorted(sq.EXPORTS) == names
    L = sq.load()
    for n in names:
        assert getattr(L, n) is not None


def test_status_strings(sq):
    for code, name in sq.STATUS_NAMES.items():
        assert sq.sq_status_string(code) == name


def _params(sq, bits=4, ng=4, mode=0):
    return sq.Params.make(bits, ng, mode)


def test_size_queries(sq):
    p = _params(sq, 4, 4)
    # layout words: 32 header + appended-column list + one descriptor per channel
    nb, ld = sq.sq_grad_layout_size(100, p)
    assert nb == (32 + 100) * 4 and ld == 112  # b=4, N_G=4: every shift fits one window, nothing appended
    p6 = _params(sq, 6, 4)
    nb, ld = sq.sq_grad_layout_size(100, p6)  # b=6: at most roundup(100, 64) + 64 * 3 appended columns
    assert nb == (32 + 320 + 100) * 4 and ld == 128 + 320
    p8 = _params(sq, 8, 4)
    nb, ld = sq.sq_grad_layout_size(64, p8)   # b=8: one window per shift
    assert nb == (32 + 256 + 64) * 4 and ld == 64 + 256
    assert sq.sq_gemm_dgrad_workspace_size(10, 100, 30, p) == 0
    assert sq.sq_gemm_dgrad_workspace_size(10, 100, 30, p6) == 30 * 320 + (256 - (30 * 320) % 256) % 256
    assert sq.sq_quantize_grad_workspace_size(10, 100, p) == 1024   # one slab of maxima + ranges
    assert sq.sq_quantize_tensor_workspace_size(10, 3) == 256


def _raw(sq):
    return sq.load()


def test_invalid_params_rejected(sq):
    L = _raw(sq)
    nb, ld = ct.c_size_t(0), ct.c_int64(0)
    for bits, ng, mode in [(1, 4, 0), (9, 4, 0), (4, 0, 0), (4, 9, 0), (4, 4, 2)]:
        p = sq.Params.make(bits, ng, mode)
        assert L.sq_grad_layout_size(64, ct.byref(p), ct.byref(nb), ct.byref(ld)) == 1
        assert sq.sq_last_error()
        assert L.sq_last_error_string().decode() == sq.sq_last_error()
    p = sq.Params.make(4, 4, 0)
    p.layout = 2
    assert L.sq_grad_layout_size(64, ct.byref(p), ct.byref(nb), ct.byref(ld)) == 1
    assert L.sq_grad_layout_size(64, None, ct.byref(nb), ct.byref(ld)) == 1


def test_quantize_grad_validation_no_launch(sq):
    L = _raw(sq)
    p = sq.Params.make(4, 4, 0)
    fake = ct.c_void_p(0x100000)   # 16-byte aligned, never dereferenced on the host
    # NULL dY
    assert L.sq_quantize_grad(None, 8, 8, 8, ct.byref(p), fake, 16, fake, 16, fake, fake, fake, fake, 4096,
                              None) == 1
    # ld_dY < C
    assert L.sq_quantize_grad(fake, 8, 8, 4, ct.byref(p), fake, 16, fake, 16, fake, fake, fake, fake, 4096,
                              None) == 1
    # ld_fold not a multiple of 16
    assert L.sq_quantize_grad(fake, 8, 8, 8, ct.byref(p), fake, 24, fake, 16, fake, fake, fake, fake, 4096,
                              None) == 1
    # misaligned code pointer
    assert L.sq_quantize_grad(fake, 8, 8, 8, ct.byref(p), ct.c_void_p(0x100008), 16, fake, 16, fake, fake,
                              fake, fake, 4096, None) == 1
    # workspace too small
    assert L.sq_quantize_grad(fake, 8, 8, 8, ct.byref(p), fake, 16, fake, 16, fake, fake, fake, fake, 16,
                              None) == 4
    # negative sizes
    assert L.sq_quantize_grad(fake, -1, 8, 8, ct.byref(p), fake, 16, fake, 16, fake, fake, fake, fake, 4096,
                              None) == 1
    assert "workspace" in sq.sq_last_error() or "dimensions" in sq.sq_last_error()


def test_quantize_grad_noalloc_validation_no_launch(sq):
    # the same synchronous checks as sq_quantize_grad, then the fixed-scratch
    # limit, all before any HIP call
    L = _raw(sq)
    p = sq.Params.make(6, 4, 1)
    fake = ct.c_void_p(0x100000)
    assert L.sq_quantize_grad_noalloc(None, 8, 8, 8, ct.byref(p), fake, 16, fake, 16, fake, fake, fake, None) == 1
    assert L.sq_quantize_grad_noalloc(fake, 8, 8, 4, ct.byref(p), fake, 16, fake, 16, fake, fake, fake, None) == 1
    assert L.sq_quantize_grad_noalloc(fake, 8, 8, 8, ct.byref(p), fake, 24, fake, 16, fake, fake, fake, None) == 1
    # a gradient whose quantizer scratch exceeds the fixed 1 MiB array
    M, C = 1 << 16, 1 << 18
    need = sq.sq_quantize_grad_workspace_size(M, C, p)
    assert need > 1 << 20
    _, ld = sq.sq_grad_layout_size(C, p)
    st = L.sq_quantize_grad_noalloc(fake, M, C, C, ct.byref(p), fake, ld, fake, M, fake, fake, fake, None)
    assert st == 4 and "sq_quantize_grad_noalloc" in sq.sq_last_error()
    # the large linear layer's gradient fits
    assert sq.sq_quantize_grad_workspace_size(8192, 11008, p) <= 1 << 20


def test_overflow_risk_rejected(sq):
    L = _raw(sq)
    fake = ct.c_void_p(0x100000)
    # dgrad: C_out * Q * 2^(N_G-1) * 128 >= 2^31 with b = 8, N_G = 8
    p = sq.Params.make(8, 8, 0)
    st = L.sq_gemm_dgrad(fake, 2048, fake, fake, fake, fake, 2048, fake, 4, 1100, 8, ct.byref(p), None, 0,
                         fake, 8, fake, 1 << 30, None)
    assert st == 2 and "overflow" in sq.sq_last_error()
    # wgrad: M * Q * 128 >= 2^31 with b = 8
    p = sq.Params.make(8, 4, 0)
    st = L.sq_gemm_wgrad(fake, 1 << 18, fake, fake, fake, 1 << 18, fake, 140000, 4, 4, ct.byref(p), None, 0,
                         fake, 4, fake, 1 << 30, None)
    assert st == 2
    # one row fewer than the bound is accepted by the range check (then fails on NULL scales)
    st = L.sq_gemm_wgrad(fake, 1 << 18, fake, None, fake, 1 << 18, fake, 130000, 4, 4, ct.byref(p), None, 0,
                         fake, 4, fake, 1 << 30, None)
    assert st == 1


def test_gemm_validation(sq):
    L = _raw(sq)
    fake = ct.c_void_p(0x100000)
    p = sq.Params.make(4, 4, 0)
    # both outputs NULL
    assert L.sq_gemm_wgrad(fake, 64, fake, fake, fake, 64, fake, 64, 4, 4, ct.byref(p), None, 0, None, 0,
                           fake, 0, None) == 1
    # xq_t ld smaller than M
    assert L.sq_gemm_wgrad(fake, 64, fake, fake, fake, 32, fake, 64, 4, 4, ct.byref(p), None, 0, fake, 4,
                           fake, 0, None) == 1
    # dgrad: wq_t ld smaller than C_out
    assert L.sq_gemm_dgrad(fake, 64, fake, fake, fake, fake, 16, fake, 8, 40, 8, ct.byref(p), None, 0,
                           fake, 8, fake, 0, None) == 1
    # dequant: bad kind
    assert L.sq_dequant(fake, 4, 4, 4, 7, fake, fake, fake, 4, fake, 4, None) == 1


def test_python_binding_has_no_fallback(sq, monkeypatch, tmp_path):
    # a missing library is an import-time error, never a silent CPU path
    monkeypatch.setattr(sq, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(sq, "_lib", None)
    with pytest.raises(ImportError):
        sq.load()


def test_l1bn_validation_no_launch(sq):
    L = _raw(sq)
    fake = ct.c_void_p(0x100000)
    n = ct.c_int64(0)
    nb = ct.c_size_t(0)
    p = sq.Params.make(8, 4, 0)
    # M must be in [1, 2^24]
    assert L.sq_l1bn_range_slabs(0, 64, ct.byref(n)) == 1
    assert L.sq_l1bn_range_slabs((1 << 24) + 1, 64, ct.byref(n)) == 3
    assert L.sq_l1bn_range_slabs(200704, 64, ct.byref(n)) == 0 and 1 <= n.value <= 1024
    assert L.sq_l1bn_forward_workspace_size(100, 64, ct.byref(nb)) == 0 and nb.value > 0
    assert L.sq_l1bn_backward_workspace_size(100, 64, ct.byref(p), ct.byref(nb)) == 0 and nb.value >= 100 * 64
    # forward: ld of the codes not a multiple of 16, NULL gamma, small workspace
    assert L.sq_l1bn_forward(fake, 8, 8, 8, fake, fake, fake, fake, 8, fake, fake, fake, 4096, None) == 1
    assert L.sq_l1bn_forward(fake, 8, 8, 16, fake, None, fake, fake, 8, fake, fake, fake, 4096, None) == 1
    assert L.sq_l1bn_forward(fake, 8, 8, 16, fake, fake, fake, fake, 8, fake, fake, fake, 16, None) == 4
    # backward: bad params, misaligned ranges, workspace not 256-byte aligned
    bad = sq.Params.make(9, 4, 0)
    assert L.sq_l1bn_backward(fake, 8, 8, 8, ct.byref(bad), fake, 16, fake, fake, fake, 8, fake, fake, fake,
                              fake, None, fake, 1 << 20, None) == 1
    assert L.sq_l1bn_backward(fake, 8, 8, 8, ct.byref(p), fake, 16, fake, fake, fake, 8, fake, fake, fake,
                              fake, ct.c_void_p(0x100002), fake, 1 << 20, None) == 1
    assert L.sq_l1bn_backward(fake, 8, 8, 8, ct.byref(p), fake, 16, fake, fake, fake, 8, fake, fake, fake,
                              fake, None, ct.c_void_p(0x100010), 1 << 20, None) == 1


def test_quantize_from_ranges_validation_no_launch(sq):
    L = _raw(sq)
    fake = ct.c_void_p(0x100000)
    p = sq.Params.make(4, 4, 0)
    # NULL ranges, zero slabs
    assert L.sq_quantize_grad_from_ranges(fake, 8, 8, 8, ct.byref(p), None, 1, fake, 16, fake, 16, fake, fake,
                                          fake, fake, 4096, None) == 1
    assert L.sq_quantize_grad_from_ranges(fake, 8, 8, 8, ct.byref(p), fake, 0, fake, 16, fake, 16, fake, fake,
                                          fake, fake, 4096, None) == 1
    assert L.sq_quantize_grad_from_ranges(fake, 8, 8, 8, ct.byref(p), fake, 1, fake, 16, fake, 16, fake, fake,
                                          fake, fake, 16, None) == 4


def test_conv_wgrad_and_ranged_dgrad_validation_no_launch(sq):
    L = _raw(sq)
    fake = ct.c_void_p(0x100000)
    p = sq.Params.make(4, 4, 0)
    rows, ld, qld = ct.c_int64(0), ct.c_int64(0), ct.c_int64(0)
    # padded grid of the ResNet-18 layer: 58 rows x 64 columns per image
    assert L.sq_conv_wgrad_layout(64, 56, 56, 64, 3, 3, 1, 1, ct.byref(rows), ct.byref(ld), ct.byref(qld)) == 0
    # one input copy: C_in rows, the grid plus (KH - 1) Wp + 64 zero columns
    assert rows.value == 64 and qld.value == 64 * 58 * 64 and ld.value == qld.value + 2 * 64 + 64
    # padding >= window, window larger than the input
    assert L.sq_conv_wgrad_layout(1, 5, 5, 8, 3, 3, 3, 1, ct.byref(rows), ct.byref(ld), ct.byref(qld)) == 1
    assert L.sq_conv_wgrad_layout(1, 1, 5, 8, 3, 3, 0, 1, ct.byref(rows), ct.byref(ld), ct.byref(qld)) == 1
    nb = ct.c_size_t(0)
    assert L.sq_conv_wgrad_workspace_size(64, 56, 56, 64, 64, 3, 3, 1, 1, ct.byref(p), ct.byref(nb)) == 0
    # too short a row of the packed input, NULL outputs
    assert L.sq_conv_wgrad(fake, qld.value, fake, fake, fake, ld.value - 16, fake, 64, 56, 56, 64, 64, 3, 3, 1, 1,
                           ct.byref(p), fake, 576, fake, 576, fake, 1 << 30, None) == 1
    assert L.sq_conv_wgrad(fake, qld.value, fake, fake, fake, ld.value, fake, 64, 56, 56, 64, 64, 3, 3, 1, 1,
                           ct.byref(p), None, 0, None, 0, fake, 1 << 30, None) == 1
    # quantize onto the padded grid: ld of the padded codes too small
    assert L.sq_quantize_grad_conv(fake, 2, 8, 8, 64, 64, 3, 3, 1, 1, ct.byref(p), fake, 64, fake, 64, fake, fake,
                                   fake, fake, 1 << 20, None) == 1
    # ranged dgrad: slab count and required dX
    n = ct.c_int64(0)
    assert L.sq_gemm_dgrad_range_slabs(1000, ct.byref(n)) == 0 and n.value == 32
    assert L.sq_gemm_dgrad_ranged(fake, 64, fake, fake, fake, fake, 64, fake, 64, 64, 64, ct.byref(p), None, 0,
                                  None, 64, fake, fake, 0, None) == 1
    assert L.sq_gemm_dgrad_ranged(fake, 64, fake, fake, fake, fake, 64, fake, 64, 64, 64, ct.byref(p), None, 0,
                                  fake, 64, None, fake, 0, None) == 1
