"""chunk_gemm_noalloc through the C-ABI: the same bits as chunk_gemm with its
queried workspace (and the oracle's, exact mode), on calls in a row that
share the library's static scratch -- a large call, then a smaller one, then
one whose fastest plan would need more than the scratch holds."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_1812_08011_amd as fp8t
from tests.gpu_util import DEV, dev, gemm, host, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fp8t.lib()
    yield


def _noalloc(A, B, M, N, K, CL, ta, tb, mode):
    """Raw C-ABI call with device addresses."""
    C = torch.full((M, N), 0xBEEF, dtype=torch.int32, device=DEV).to(torch.uint16)
    L = fp8t.lib()
    st = L.chunk_gemm_noalloc(ta, tb, M, N, K, CL, ctypes.c_void_p(A.data_ptr()),
                              A.shape[1], ctypes.c_void_p(B.data_ptr()), B.shape[1],
                              ctypes.c_void_p(C.data_ptr()), N, mode,
                              ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, fp8t.status_string(st)
    return host(C)


def _operands(rng, M, N, K, ta, tb):
    a = rng.standard_normal((M, K)).astype(np.float32)
    b = rng.standard_normal((K, N)).astype(np.float32)
    A = oracle.fp8_quantize(np.ascontiguousarray(a.T if ta else a))
    B = oracle.fp8_quantize(np.ascontiguousarray(b.T if tb else b))
    return A, B


# (M, N, K, CL, ta, tb, env): shared tiles through the scratch, then smaller
# calls, then a call whose fastest plan needs more than the scratch
CASES = [
    (512, 384, 8192, 64, 0, 0, {"FP8T_GEMM_SPLIT": "1"}),
    # fast mode: the matrix-core kernel that reads a k-contiguous copy of B
    # (made in the scratch)
    (300, 640, 2048, 64, 0, 0, {"FP8T_MFMA_TILE": "5"}),
    (200, 150, 3000, 64, 1, 0, {"FP8T_GEMM_SPLIT": "1", "FP8T_GEMM_WGS": "7"}),
    (2304, 256, 16384, 64, 1, 0, {}),
]


@pytest.mark.parametrize("mode", [fp8t.EXACT, fp8t.FAST])
def test_noalloc_matches_chunk_gemm(mode, monkeypatch):
    rng = np.random.default_rng(1300 + mode)
    for (M, N, K, CL, ta, tb, env) in CASES:
        for k in ("FP8T_GEMM_SPLIT", "FP8T_GEMM_WGS", "FP8T_MFMA_TILE"):
            monkeypatch.delenv(k, raising=False)
        for k, v in env.items():
            monkeypatch.setenv(k, v)
        A, B = _operands(rng, M, N, K, ta, tb)
        Ad, Bd = dev(A), dev(B)
        ws = fp8t.chunk_gemm_workspace_size(ta, tb, M, N, K, CL, mode)
        say(f"noalloc mode={mode} {M}x{N}x{K} CL={CL} ta={ta} tb={tb} env={env} "
            f"(chunk_gemm workspace {ws} bytes, scratch {64 << 20})")
        got = _noalloc(Ad, Bd, M, N, K, CL, ta, tb, mode)
        ref = host(gemm(Ad, Bd, M, N, K, CL, ta, tb, mode=mode))
        assert np.array_equal(got, ref), np.argwhere(got != ref)[:5]
        if mode == fp8t.EXACT and M * N * K <= 100_000_000:
            assert np.array_equal(got, oracle.chunk_gemm(A, B, CL, ta, tb))
        # a second call on the same scratch gives the same bits again
        again = _noalloc(Ad, Bd, M, N, K, CL, ta, tb, mode)
        assert np.array_equal(again, got)
