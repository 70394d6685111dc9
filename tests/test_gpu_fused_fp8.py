"""GPU parity of chunk_gemm_fp8, the GEMM whose FP16 result is rounded back to
FP8 (optionally scaled) in the same pass.  Its definition is a composition of
two pinned oracle functions: C8 = fp8_quantize(chunk_gemm(A, B), FP16 source,
scale).  Exact mode is compared with that composition bit for bit; in fast
mode C8 must equal the quantized FP16 result of the same call (and of
chunk_gemm), bit for bit, whatever the plan."""
import numpy as np
import pytest
import torch

import oracle
import paper_1812_08011_amd as fp8t
from tests.gpu_util import DEV, dev, host, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fp8t.lib()
    yield


def _operands(rng, M, N, K, ta, tb, big=False):
    a = rng.standard_normal((M, K)).astype(np.float32)
    b = rng.standard_normal((K, N)).astype(np.float32)
    if big:
        a *= np.float32(300.0)
        b *= np.float32(300.0)
    a[rng.random(a.shape) < 0.05] = 0.0
    A = oracle.fp8_quantize(np.ascontiguousarray(a.T if ta else a))
    B = oracle.fp8_quantize(np.ascontiguousarray(b.T if tb else b))
    return A, B


def run_fp8(Ad, Bd, M, N, K, CL, ta, tb, mode, scale, with_c, ldc8=None):
    lda = Ad.shape[-1]
    ldb = Bd.shape[-1]
    ldc8 = ldc8 or N
    ws_b = fp8t.chunk_gemm_fp8_workspace_size(ta, tb, M, N, K, CL, mode)
    ws = torch.empty(ws_b, dtype=torch.uint8, device=DEV) if ws_b else None
    C = torch.full((M, N), 0xABCD, dtype=torch.uint16, device=DEV) if with_c else None
    C8 = torch.full((M, ldc8), 0xA5, dtype=torch.uint8, device=DEV)
    fp8t.chunk_gemm_fp8(ta, tb, M, N, K, CL, Ad, lda, Bd, ldb, C, N, C8, ldc8, scale, mode, ws,
                        ws_b)
    C8h = host(C8)
    assert np.all(C8h[:, N:] == 0xA5)                 # padding untouched
    return (host(C) if with_c else None), C8h[:, :N]


def run_fp16(Ad, Bd, M, N, K, CL, ta, tb, mode):
    ws_b = fp8t.chunk_gemm_workspace_size(ta, tb, M, N, K, CL, mode)
    ws = torch.empty(ws_b, dtype=torch.uint8, device=DEV) if ws_b else None
    C = torch.empty((M, N), dtype=torch.uint16, device=DEV)
    fp8t.chunk_gemm(ta, tb, M, N, K, CL, Ad, Ad.shape[-1], Bd, Bd.shape[-1], C, N, mode, ws, ws_b)
    return host(C)


SHAPES = [
    # M, N, K, CL
    (130, 67, 333, 64),
    (64, 96, 4096, 32),
    (33, 47, 700, 48),
    (200, 150, 1000, 16),
]


@pytest.mark.parametrize("plan", ["auto", "shared", "tile8x8"])
@pytest.mark.parametrize("mode", [fp8t.EXACT, fp8t.FAST])
@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0)])
def test_chunk_gemm_fp8_matches_quantized_result(ta, tb, mode, plan, monkeypatch):
    if plan == "shared":
        monkeypatch.setenv("FP8T_GEMM_SPLIT", "1")
        monkeypatch.setenv("FP8T_GEMM_WGS", "5")
    if plan == "tile8x8":                   # 8 x 8 register tiles (exact mode)
        monkeypatch.setenv("FP8T_VALU_TILE", "1")
    rng = np.random.default_rng(700 + 2 * ta + tb + 10 * mode)
    for (M, N, K, CL) in SHAPES:
        A, B = _operands(rng, M, N, K, ta, tb)
        Ad, Bd = dev(A), dev(B)
        C16 = run_fp16(Ad, Bd, M, N, K, CL, ta, tb, mode)
        if mode == fp8t.EXACT:
            assert np.array_equal(C16, oracle.chunk_gemm(A, B, CL, ta, tb))
        for scale in (1.0, 1000.0, 0.125):
            ref = oracle.fp8_quantize(C16, scale)
            # a leading dimension that allows no wide stores, and one that
            # allows 4- and 8-byte stores
            for with_c, ldc8 in ((True, N + 3), (False, N + 3), (False, (N + 3) // 8 * 8 + 8)):
                say(f"chunk_gemm_fp8 mode={mode} plan={plan} ta={ta} tb={tb} {M}x{N}x{K} "
                    f"CL={CL} scale={scale} C={with_c} ldc8={ldc8}")
                Cg, C8 = run_fp8(Ad, Bd, M, N, K, CL, ta, tb, mode, scale, with_c, ldc8=ldc8)
                assert np.array_equal(C8, ref), np.argwhere(C8 != ref)[:5]
                if with_c:
                    assert np.array_equal(Cg, C16)


@pytest.mark.parametrize("mode", [fp8t.EXACT, fp8t.FAST])
def test_chunk_gemm_fp8_specials_and_saturation(mode):
    """Results beyond FP8's range saturate, Inf results give Inf codes, NaN
    results the canonical NaN code -- as fp8_quantize of the FP16 result."""
    rng = np.random.default_rng(720 + mode)
    M, N, K, CL = 70, 40, 512, 64
    A, B = _operands(rng, M, N, K, 0, 0, big=True)
    A[3, :] = 0x7B                      # rows whose sums overflow FP16
    A[7, 5] = 0x7C                      # +Inf operand
    A[9, 6] = 0x7F                      # NaN operand
    Ad, Bd = dev(A), dev(B)
    C16 = run_fp16(Ad, Bd, M, N, K, CL, 0, 0, mode)
    for scale in (1.0, 1e-3, -2.0):
        say(f"chunk_gemm_fp8 specials mode={mode} scale={scale}")
        _, C8 = run_fp8(Ad, Bd, M, N, K, CL, 0, 0, mode, scale, False)
        assert np.array_equal(C8, oracle.fp8_quantize(C16, scale))


def test_chunk_gemm_fp8_empty_k():
    """K = 0: every FP16 result is +0 and the FP8 result is Q8(0 * scale)."""
    for scale in (1.0, float("inf")):
        say(f"chunk_gemm_fp8 K=0 scale={scale}")
        C = torch.full((5, 7), 0x1234, dtype=torch.uint16, device=DEV)
        C8 = torch.full((5, 7), 0x11, dtype=torch.uint8, device=DEV)
        A = torch.zeros((5, 1), dtype=torch.uint8, device=DEV)
        B = torch.zeros((1, 7), dtype=torch.uint8, device=DEV)
        fp8t.chunk_gemm_fp8(0, 0, 5, 7, 0, 64, A, 1, B, 7, C, 7, C8, 7, scale, fp8t.EXACT)
        assert np.all(host(C) == 0)
        want = oracle.fp8_quantize(np.zeros((5, 7), np.float32), scale)
        assert np.array_equal(host(C8), want)
