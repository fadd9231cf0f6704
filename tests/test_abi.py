"""Host-side checks of libfqt.so: it loads, exports every function include/fqt.h
declares, sizes workspaces, and rejects bad arguments before any launch.
No GPU work is started here: every call below returns during validation."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fqt.h")
LIB = os.path.join(ROOT, "paper_2010_14298_amd", "libfqt.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libfqt.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fqt_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_paper_entry_points():
    names = declared_functions()
    for n in ("fqt_quantize_ptq", "fqt_quantize_psq", "fqt_quantize_bhq", "fqt_linear_backward",
              "fqt_conv_backward_im2col"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(LIB)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_exports_match_header():
    from paper_2010_14298_amd import fqt
    assert sorted(fqt.EXPORTS) == declared_functions()


def test_workspace_queries_and_argument_errors():
    from paper_2010_14298_amd import fqt
    lib = fqt.load()
    cfg = fqt.cfg_struct(qb_x=("bhq", 5, 64))
    n = lib.fqt_linear_backward_workspace(8192, 1024, 4096, ctypes.byref(cfg))
    # codes of X, W, G twice, plus stats and plan: at least the code bytes
    assert n >= 8192 * 1024 + 1024 * 4096 + 2 * 8192 * 4096
    assert lib.fqt_linear_backward_workspace(0, 1, 1, ctypes.byref(cfg)) == 0
    assert lib.fqt_quantize_workspace(fqt.FQT_BHQ, 128, 10, 64) > lib.fqt_quantize_workspace(fqt.FQT_PTQ, 128, 10, 0)
    null = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(0x1000)      # never dereferenced: validation fails first
    # NULL inputs
    rc = lib.fqt_linear_backward(null, fake, fake, 4, 4, 4, ctypes.byref(cfg), fake, fake, fake, 1 << 30, null)
    assert rc == 1
    # bits out of range
    bad = fqt.cfg_struct(qb_x=("psq", 9, 0))
    rc = lib.fqt_linear_backward(fake, fake, fake, 4, 4, 4, ctypes.byref(bad), fake, fake, fake, 1 << 30, null)
    assert rc == 1
    # a per-sample grad_W quantizer on a linear layer: its per-row scales lie on
    # the contraction axis, one sample per K step, so the layer takes the shift form
    unsup = fqt.cfg_struct(qb_w=("psq", 8, 0))
    rc = lib.fqt_linear_backward(fake, fake, fake, 4, 4, 4, ctypes.byref(unsup), fake, fake, fake, 1 << 30, null)
    assert rc == 2
    assert lib.fqt_linear_backward_workspace(4, 4, 4, ctypes.byref(unsup)) == 0
    rc = lib.fqt_linear_backward(fake, fake, fake, 4, 4, 4, ctypes.byref(fqt.cfg_struct(qb_w=("bhq", 8, 4))),
                                 fake, fake, fake, 1 << 30, null)
    assert rc == 2
    # App. D's adaptive groups (block size 0) score every number of groups: at most 65536 rows
    rc = lib.fqt_linear_backward(fake, fake, fake, 70000, 4, 4, ctypes.byref(fqt.cfg_struct(qb_x=("bhq", 5, 0))),
                                 fake, fake, fake, 1 << 30, null)
    assert rc == 2
    assert lib.fqt_bhq_adaptive_groups(fake, 70000, 4, 5, fake, null, fake, 1 << 30, null) == 2
    assert lib.fqt_bhq_adaptive_groups(fake, 40, 4, 9, fake, null, fake, 1 << 30, null) == 1
    assert lib.fqt_bhq_adaptive_groups(fake, 40, 4, 5, null, null, fake, 1 << 30, null) == 1
    assert lib.fqt_bhq_adaptive_groups(fake, 40, 4, 5, fake, null, fake, 16, null) == 4
    assert lib.fqt_bhq_adaptive_workspace(40, 4) > lib.fqt_quantize_workspace(fqt.FQT_BHQ, 40, 4, 64)
    # a negative block size
    rc = lib.fqt_linear_backward(fake, fake, fake, 4, 4, 4, ctypes.byref(fqt.cfg_struct(qb_x=("bhq", 5, -1))),
                                 fake, fake, fake, 1 << 30, null)
    assert rc == 1
    # workspace too small / missing
    rc = lib.fqt_linear_backward(fake, fake, fake, 4, 4, 4, ctypes.byref(cfg), fake, fake, fake, 16, null)
    assert rc == 4
    rc = lib.fqt_linear_backward(fake, fake, fake, 4, 4, 4, ctypes.byref(cfg), fake, fake, null, 1 << 30, null)
    assert rc == 4
    # quantizer arguments
    qt = fqt.QTensor(0x1000, 0x1000, 0x1000, 0, 0, 0)
    assert lib.fqt_quantize_psq(fake, 0, 4, 8, 0, 0, ctypes.byref(qt), fake, 1 << 30, null) == 1
    assert lib.fqt_quantize_psq(fake, 4, 4, 0, 0, 0, ctypes.byref(qt), fake, 1 << 30, null) == 1
    assert lib.fqt_quantize_bhq(fake, 4, 4, 5, 64, 0, 0, ctypes.byref(qt), fake, 1 << 30, null) == 1   # no perm
    assert lib.fqt_gemm_s8s8_s64(fake, fake, 4, 4, 8, 4, 8, fake, fake, 1 << 30, null) == 1            # lda < K
    assert lib.fqt_gemm_s4s4_bf6(fake, fake, 4, 4, 8, 4, 8, fake, fake, 1 << 30, null) == 1            # lda < K
    assert lib.fqt_gemm_s4s4_bf6(fake, fake, 4, 4, 8, 8, 8, fake, fake, 16, null) == 4
    assert lib.fqt_gemm_s4s4_bf6_workspace(0, 4, 4) == 0
    ops = ctypes.c_double(0)
    assert lib.fqt_probe_mfma_i8(0, fake, ctypes.byref(ops), null) == 1
    assert lib.fqt_probe_copy(fake, fake, 24, null) == 1
    # packed rows: 96 bytes per 128 codes
    assert lib.fqt_gemm_s4s4_bf6_workspace(128, 128, 4096) >= 2 * 128 * 3072 + 128 * 128 * 4
    assert lib.fqt_status_str(3) == b"non-finite input or range overflow"
    # layer forward: bits, relu flag, workspace
    assert lib.fqt_linear_forward_workspace(0, 4, 4) == 0
    assert lib.fqt_linear_forward_workspace(8192, 1024, 4096) >= 8192 * 1024 + 4096 * 1024
    assert lib.fqt_linear_forward(null, fake, 4, 8, 3, 8, 8, 0, fake, fake, 1 << 30, null) == 1
    assert lib.fqt_linear_forward(fake, fake, 4, 8, 3, 9, 8, 0, fake, fake, 1 << 30, null) == 1
    assert lib.fqt_linear_forward(fake, fake, 4, 8, 3, 8, 8, 2, fake, fake, 1 << 30, null) == 1
    assert lib.fqt_linear_forward(fake, fake, 4, 8, 3, 8, 8, 1, fake, fake, 16, null) == 4
    assert lib.fqt_linear_forward(fake, fake, 4, 8, 3, 8, 8, 1, fake, null, 1 << 30, null) == 4
    # relu_input: 0 or 1; the conv backward has no masked epilogue
    relu2 = fqt.cfg_struct(relu_input=True)
    relu2.relu_input = 2
    rc = lib.fqt_linear_backward(fake, fake, fake, 4, 4, 4, ctypes.byref(relu2), fake, fake, fake, 1 << 30, null)
    assert rc == 1
    # (o = 16 passes the shape checks, so the rejection comes from the
    # configuration, before anything is launched on the fake pointers)
    sh = fqt.conv_shape(2, 4, 8, 8, 16, 3, 3, 1, 1)
    assert lib.fqt_conv_backward_workspace(ctypes.byref(sh), ctypes.byref(cfg)) > 0
    rc = lib.fqt_conv_backward_im2col(fake, fake, fake, ctypes.byref(sh), ctypes.byref(fqt.cfg_struct(relu_input=True)),
                                      fake, fake, fake, 1 << 30, null)
    assert rc == 2
    rc = lib.fqt_conv_backward_im2col(fake, fake, fake, ctypes.byref(sh),
                                      ctypes.byref(fqt.cfg_struct(qb_w=("shift", 4, 0))), fake, fake, fake, 1 << 30, null)
    assert rc == 2
    # a per-sample grad_W quantizer on a conv: one K block of 128-byte stages
    # per sample (8 x 8 outputs pad to 128), an int32 partial per sample
    psq1 = fqt.cfg_struct(qb_w=("psq", 8, 0))
    ws_psq = lib.fqt_conv_backward_workspace(ctypes.byref(sh), ctypes.byref(psq1))
    assert ws_psq >= 2 * 16 * 9 * 4 * 4 + 16 * 2 * 128 + 9 * 4 * 2 * 128
    # stride-1 layers with dense enough grids contract over shifted copies of
    # the activation codes, not an im2col matrix: the 56 x 56 batch-128
    # layer's whole workspace is below its im2col matrix alone
    l56 = fqt.conv_shape(128, 64, 56, 56, 64, 3, 3, 1, 1)
    for q in (cfg, psq1):
        assert lib.fqt_conv_backward_workspace(ctypes.byref(l56), ctypes.byref(q)) < 9 * 64 * 128 * 56 * 56
    # more output pixels than one int32-exact K block holds
    big = fqt.conv_shape(1, 16, 260, 260, 16, 1, 1, 1, 0)
    rc = lib.fqt_conv_backward_im2col(fake, fake, fake, ctypes.byref(big), ctypes.byref(psq1), fake, fake, fake,
                                      1 << 40, null)
    assert rc == 2
