"""The C-ABI library (include/fp8train.h) loads, exports every declared entry
point, and rejects invalid arguments before touching the GPU.

No compute call is made here: each call below fails validation, which the
library checks before any HIP call, so these run without a GPU.
"""
import ctypes
import os
import re

import pytest

import paper_1812_08011_amd as fp8t

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fp8train.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*([a-z_0-9]+)\s*\(", text, flags=re.M)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(fp8t.LIB_PATH):
        pytest.skip("libfp8train.so is not built")
    return fp8t.lib()


def test_header_declares_the_boundary():
    assert declared_functions() == sorted([
        "fp8_quantize", "fp16_quantize", "chunk_gemm", "chunk_gemm_workspace_size",
        "chunk_gemm_noalloc",
        "chunk_gemm_fp8", "chunk_gemm_fp8_workspace_size",
        "chunk_gemm_sr", "chunk_gemm_sr_workspace_size", "adam_update",
        "chunk_gemm_p16", "chunk_gemm_p16_workspace_size",
        "relu_codes", "relu_backward_fp8", "mse_grad_fp16",
        "conv2d_fwd_fp8", "conv2d_wgrad_fp8", "conv2d_workspace_size", "col2im_fp16",
        "sr_weight_update", "fp8t_status_string"])


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    assert fp8t.status_string(0) == "ok"
    assert "invalid" in fp8t.status_string(-1)
    assert "workspace" in fp8t.status_string(-2)
    assert fp8t.status_string(12345) == "unknown status"


FAKE = 0x10000        # never dereferenced: validation fails first


def test_fp8_quantize_rejects(lib):
    assert lib.fp8_quantize(FAKE, 0, 1.0, FAKE, -1, None) == fp8t.EINVAL
    assert lib.fp8_quantize(FAKE, 7, 1.0, FAKE, 10, None) == fp8t.EINVAL
    assert lib.fp8_quantize(None, 0, 1.0, FAKE, 10, None) == fp8t.EINVAL
    assert lib.fp8_quantize(FAKE, 0, 1.0, None, 10, None) == fp8t.EINVAL
    assert lib.fp8_quantize(None, 0, 1.0, None, 0, None) == fp8t.OK     # empty: no-op
    assert lib.fp16_quantize(None, FAKE, 5, None) == fp8t.EINVAL
    assert lib.fp16_quantize(FAKE, FAKE, -5, None) == fp8t.EINVAL


def _gemm(lib, **kw):
    a = dict(ta=0, tb=0, M=4, N=4, K=4, CL=2, A=FAKE, lda=4, B=FAKE, ldb=4, C=FAKE, ldc=4,
             mode=0, ws=None, wsb=0)
    a.update(kw)
    return lib.chunk_gemm(a["ta"], a["tb"], a["M"], a["N"], a["K"], a["CL"], a["A"], a["lda"],
                          a["B"], a["ldb"], a["C"], a["ldc"], a["mode"], a["ws"], a["wsb"], None)


def test_chunk_gemm_rejects(lib):
    E = fp8t.EINVAL
    assert _gemm(lib, CL=0) == E
    assert _gemm(lib, CL=-3) == E
    assert _gemm(lib, M=-1) == E
    assert _gemm(lib, K=-1) == E
    assert _gemm(lib, ta=2) == E
    assert _gemm(lib, tb=-1) == E
    assert _gemm(lib, mode=2) == E
    assert _gemm(lib, lda=3) == E                       # lda < K
    assert _gemm(lib, ta=1, M=8, lda=4) == E            # lda < M
    assert _gemm(lib, ldb=3) == E                       # ldb < N
    assert _gemm(lib, tb=1, K=8, ldb=4, lda=8) == E     # ldb < K
    assert _gemm(lib, ldc=3) == E
    assert _gemm(lib, A=None) == E
    assert _gemm(lib, B=None) == E
    assert _gemm(lib, C=None) == E
    assert _gemm(lib, M=2 ** 31) == E                   # beyond 32-bit dimensions
    assert _gemm(lib, N=2 ** 31 - 4096, ldb=2 ** 31, ldc=2 ** 31) == E  # no room for tile ends
    assert _gemm(lib, K=2 ** 31 - 4096, lda=2 ** 31) == E
    assert _gemm(lib, M=0) == fp8t.OK                   # empty output: no-op
    assert _gemm(lib, N=0, C=None) == fp8t.OK


def test_chunk_gemm_noalloc_rejects(lib):
    """Validation comes before the scratch's device address is taken, so the
    rejections need no GPU."""
    def call(**kw):
        a = dict(ta=0, tb=0, M=4, N=4, K=4, CL=2, A=FAKE, lda=4, B=FAKE, ldb=4, C=FAKE, ldc=4,
                 mode=0)
        a.update(kw)
        return lib.chunk_gemm_noalloc(a["ta"], a["tb"], a["M"], a["N"], a["K"], a["CL"], a["A"],
                                      a["lda"], a["B"], a["ldb"], a["C"], a["ldc"], a["mode"],
                                      None)
    E = fp8t.EINVAL
    for kw in (dict(CL=0), dict(M=-1), dict(ta=2), dict(mode=3), dict(lda=3), dict(ldb=3),
               dict(ldc=3), dict(A=None), dict(C=None), dict(M=2 ** 31)):
        assert call(**kw) == E, kw
    assert call(M=0) == fp8t.OK


def _gemm8(lib, **kw):
    a = dict(ta=0, tb=0, M=4, N=4, K=4, CL=2, A=FAKE, lda=4, B=FAKE, ldb=4, C=FAKE, ldc=4,
             C8=FAKE, ldc8=4, scale=1.0, mode=0, ws=None, wsb=0)
    a.update(kw)
    return lib.chunk_gemm_fp8(a["ta"], a["tb"], a["M"], a["N"], a["K"], a["CL"], a["A"],
                              a["lda"], a["B"], a["ldb"], a["C"], a["ldc"], a["C8"], a["ldc8"],
                              a["scale"], a["mode"], a["ws"], a["wsb"], None)


def test_chunk_gemm_fp8_rejects(lib):
    E = fp8t.EINVAL
    assert _gemm8(lib, C8=None) == E
    assert _gemm8(lib, ldc8=3) == E
    assert _gemm8(lib, ldc=3) == E                      # C given with ldc < N
    assert _gemm8(lib, CL=0) == E
    assert _gemm8(lib, mode=5) == E
    assert _gemm8(lib, lda=3) == E
    assert _gemm8(lib, A=None) == E
    assert _gemm8(lib, ws=None, wsb=64) == E            # workspace size without a pointer
    assert _gemm8(lib, M=0) == fp8t.OK
    assert _gemm(lib, ws=None, wsb=64) == E


def _gemm_sr(lib, **kw):
    a = dict(ta=0, tb=0, M=4, N=4, K=4, CL=2, A=FAKE, lda=4, B=FAKE, ldb=4, C=FAKE, ldc=4,
             seed=1, offset=0, ws=None, wsb=0)
    a.update(kw)
    return lib.chunk_gemm_sr(a["ta"], a["tb"], a["M"], a["N"], a["K"], a["CL"], a["A"], a["lda"],
                             a["B"], a["ldb"], a["C"], a["ldc"], a["seed"], a["offset"], a["ws"],
                             a["wsb"], None)


def test_chunk_gemm_sr_rejects(lib):
    E = fp8t.EINVAL
    assert _gemm_sr(lib, CL=0) == E
    assert _gemm_sr(lib, M=-1) == E
    assert _gemm_sr(lib, ta=3) == E
    assert _gemm_sr(lib, lda=3) == E
    assert _gemm_sr(lib, ldb=3) == E
    assert _gemm_sr(lib, ldc=3) == E
    assert _gemm_sr(lib, C=None) == E
    assert _gemm_sr(lib, B=None) == E
    assert _gemm_sr(lib, offset=2 ** 31) == E
    assert _gemm_sr(lib, K=2 ** 31) == E
    assert _gemm_sr(lib, ws=None, wsb=64) == E
    assert _gemm_sr(lib, M=0) == fp8t.OK
    assert fp8t.chunk_gemm_sr_workspace_size(0, 0, 4, 4, 4, 0) == 0


def test_chunk_gemm_p16_rejects(lib):
    E = fp8t.EINVAL
    f = lib.chunk_gemm_p16

    def call(**kw):
        a = dict(ta=0, tb=0, M=4, N=4, K=4, CL=2, A=FAKE, lda=4, B=FAKE, ldb=4, C=FAKE, ldc=4,
                 ws=None, wsb=0)
        a.update(kw)
        return f(a["ta"], a["tb"], a["M"], a["N"], a["K"], a["CL"], a["A"], a["lda"], a["B"],
                 a["ldb"], a["C"], a["ldc"], a["ws"], a["wsb"], None)
    assert call(CL=0) == E
    assert call(tb=2) == E
    assert call(lda=3) == E
    assert call(ldc=3) == E
    assert call(A=None) == E
    assert call(ws=None, wsb=8) == E
    assert call(N=0) == fp8t.OK
    assert fp8t.chunk_gemm_p16_workspace_size(0, 0, 4, 4, 4, 0) == 0


def test_elementwise_rejects(lib):
    E = fp8t.EINVAL
    assert lib.relu_codes(FAKE, 7, FAKE, 4, None) == E
    assert lib.relu_codes(FAKE, 8, FAKE, -1, None) == E
    assert lib.relu_codes(None, 16, FAKE, 4, None) == E
    assert lib.relu_codes(None, 16, None, 0, None) == fp8t.OK
    assert lib.relu_backward_fp8(FAKE, None, FAKE, 4, 1.0, None) == E
    assert lib.relu_backward_fp8(FAKE, FAKE, FAKE, -2, 1.0, None) == E
    assert lib.mse_grad_fp16(FAKE, FAKE, None, 4, 1.0, None) == E
    assert lib.mse_grad_fp16(None, None, None, 0, 1.0, None) == fp8t.OK


def test_conv_rejects(lib):
    E = fp8t.EINVAL

    def fwd(**kw):
        a = dict(X=FAKE, N=2, H=5, W=5, C=4, KH=3, KW=3, pad=1, stride=1, Wt=FAKE, Cout=8, CL=64,
                 Y=FAKE, ldy=8, ws=None, wsb=0)
        a.update(kw)
        return lib.conv2d_fwd_fp8(a["X"], a["N"], a["H"], a["W"], a["C"], a["KH"], a["KW"],
                                  a["pad"], a["stride"], a["Wt"], a["Cout"], a["CL"], a["Y"],
                                  a["ldy"], a["ws"], a["wsb"], None)
    for bad in (dict(N=-1), dict(H=0), dict(C=0), dict(KH=0), dict(stride=0), dict(pad=-1),
                dict(KH=8), dict(Cout=-1), dict(CL=0), dict(X=None), dict(Wt=None),
                dict(Y=None), dict(ldy=7), dict(ws=None, wsb=16),
                dict(Cout=2 ** 31 - 4096, ldy=2 ** 31)):
        assert fwd(**bad) == E, bad
    assert fwd(N=0) == fp8t.OK
    assert fwd(Cout=0) == fp8t.OK
    assert lib.conv2d_wgrad_fp8(FAKE, 2, 5, 5, 4, 3, 3, 1, 1, FAKE, 8, 64, FAKE, 7, None, 0,
                                None) == E
    assert fp8t.conv2d_workspace_size(2, 2, 5, 5, 4, 3, 3, 1, 1, 8, 64) == 0
    assert fp8t.conv2d_workspace_size(0, 2, 5, 5, 4, 3, 3, 1, 0, 8, 64) == 0
    assert lib.col2im_fp16(FAKE, 2, 5, 5, 4, 3, 3, 1, 0, FAKE, None) == E
    assert lib.col2im_fp16(None, 2, 5, 5, 4, 3, 3, 1, 1, FAKE, None) == E
    assert lib.col2im_fp16(None, 0, 5, 5, 4, 3, 3, 1, 1, None, None) == fp8t.OK


def test_workspace_size_without_a_device(lib):
    """The query plans for the current device; with none it reports 0, and 0
    for invalid arguments."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("a device is present")
    assert fp8t.chunk_gemm_workspace_size(0, 0, 128, 128, 1024, 64, 0) == 0
    assert fp8t.chunk_gemm_fp8_workspace_size(0, 0, 128, 128, 1024, 64, 0) == 0
    assert fp8t.chunk_gemm_workspace_size(0, 0, 128, 128, 1024, 0, 0) == 0
    assert fp8t.chunk_gemm_sr_workspace_size(0, 0, 128, 128, 1024, 64) == 0


def test_sr_weight_update_rejects(lib):
    E = fp8t.EINVAL
    f = lib.sr_weight_update
    assert f(FAKE, FAKE, None, None, 10, 0.1, 0.9, 0.0, 1, 0, None) == E   # momentum, no v
    assert f(FAKE, FAKE, FAKE, None, -1, 0.1, 0.9, 0.0, 1, 0, None) == E
    assert f(None, FAKE, None, None, 10, 0.1, 0.0, 0.0, 1, 0, None) == E
    assert f(FAKE, None, None, None, 10, 0.1, 0.0, 0.0, 1, 0, None) == E
    assert f(None, None, None, None, 0, 0.1, 0.0, 0.0, 1, 0, None) == fp8t.OK


def test_adam_update_rejects(lib):
    E = fp8t.EINVAL
    f = lib.adam_update
    args = [FAKE, FAKE, FAKE, FAKE, None, 10, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1, 1, 0, None]
    assert f(*args[:11], 0, *args[12:]) == E                  # t = 0
    assert f(*args[:5], -1, *args[6:]) == E                   # n < 0
    for k in range(4):                                        # NULL w, g, m, v
        a = list(args)
        a[k] = None
        assert f(*a) == E
    assert f(None, None, None, None, None, 0, *args[6:]) == fp8t.OK


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    monkeypatch.setattr(fp8t, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(fp8t, "_lib", None)
    with pytest.raises(RuntimeError, match="not built"):
        fp8t.lib()


def test_product_path_does_not_import_the_oracle():
    pkg = os.path.dirname(fp8t.__file__)
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in text and "from oracle" not in text, f
                assert "liboracle" not in text and "oracle.h" not in text, f
