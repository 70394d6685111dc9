"""GPU parity of chunk_gemm_sr (stochastic rounding after every FP16
addition) with the oracle, bit for bit: every layout, chunk lengths that
divide K or leave a ragged chunk, CL = 1 and CL >= K, tiles processed whole
or shared out over workgroups (the random bits belong to (i, j, k), so the
plan cannot change the result), specials and degenerate sizes."""
import numpy as np
import pytest
import torch

import oracle
import paper_1812_08011_amd as fp8t
import workloads
from tests.gpu_util import DEV, dev, host, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fp8t.lib()
    yield


def sr_gemm(Ad, Bd, M, N, K, CL, ta, tb, seed, offset=0, use_ws=True):
    lda = Ad.shape[-1]
    ldb = Bd.shape[-1]
    wb = fp8t.chunk_gemm_sr_workspace_size(ta, tb, M, N, K, CL) if use_ws else 0
    ws = torch.empty(wb, dtype=torch.uint8, device=DEV) if wb else None
    C = torch.full((M, N), 0xABCD, dtype=torch.uint16, device=DEV)
    fp8t.chunk_gemm_sr(ta, tb, M, N, K, CL, Ad, lda, Bd, ldb, C, N, seed, offset, ws, wb)
    return host(C)


def operands(rng, M, N, K, ta, tb, scale=1.0):
    a = (rng.standard_normal((M, K)) * scale).astype(np.float32)
    b = (rng.standard_normal((K, N)) * scale).astype(np.float32)
    a[rng.random(a.shape) < 0.05] = 0.0
    A = oracle.fp8_quantize(np.ascontiguousarray(a.T if ta else a))
    B = oracle.fp8_quantize(np.ascontiguousarray(b.T if tb else b))
    return A, B


SHAPES = [
    # M, N, K, CL
    (130, 67, 333, 64),
    (64, 96, 1000, 7),
    (33, 47, 700, 700),
    (70, 150, 600, 1),
    (5, 3, 17, 4),
    (128, 64, 4096, 256),
]


@pytest.mark.parametrize("plan", ["auto", "shared", "no_ws"])
@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_sr_gemm_matches_oracle(ta, tb, plan, monkeypatch):
    if plan == "shared":
        monkeypatch.setenv("FP8T_GEMM_SPLIT", "1")
        monkeypatch.setenv("FP8T_GEMM_WGS", "7")
    rng = np.random.default_rng(800 + 2 * ta + tb)
    for i, (M, N, K, CL) in enumerate(SHAPES):
        A, B = operands(rng, M, N, K, ta, tb, scale=4.0)
        seed, offset = 1000 + i, 3 * i
        say(f"chunk_gemm_sr plan={plan} ta={ta} tb={tb} {M}x{N}x{K} CL={CL} seed={seed}")
        got = sr_gemm(dev(A), dev(B), M, N, K, CL, ta, tb, seed, offset, use_ws=plan != "no_ws")
        ref = oracle.chunk_gemm_sr(A, B, CL, ta, tb, seed=seed, offset=offset)
        assert np.array_equal(got, ref), (M, N, K, CL, np.argwhere(got != ref)[:5])


def test_sr_gemm_fig3b_rows():
    """Fig. 3(b) on the GPU: the same mean-1 vector in 40 rows (different
    random bits per row), CL = K and CL = 64, against the oracle."""
    L, R = 12000, 40
    a = oracle.fp8_quantize(workloads.accumulation_vector(L))
    A = np.ascontiguousarray(np.broadcast_to(a[None, :], (R, L)))
    B = np.full((L, 1), 0x3C, np.uint8)
    exact = float(np.sum(oracle.p8_value(a)))
    for CL in (L, 64):
        say(f"chunk_gemm_sr fig3b rows CL={CL}")
        got = sr_gemm(dev(A), dev(B), R, 1, L, CL, 0, 0, seed=31)
        assert np.array_equal(got, oracle.chunk_gemm_sr(A, B, CL, seed=31))
        v = oracle.p16_value(got)[:, 0]
        assert abs(float(np.mean(v)) - exact) / exact < 0.02


def test_sr_gemm_specials():
    rng = np.random.default_rng(830)
    M, N, K, CL = 70, 40, 512, 64
    A, B = operands(rng, M, N, K, 0, 0, scale=300.0)
    A[3, :] = 0x7B                      # sums overflow FP16
    A[7, 5] = 0x7C                      # +Inf operand
    A[9, 6] = 0x7F                      # NaN operand
    A[11, 1] = 0xFC                     # -Inf operand
    say("chunk_gemm_sr specials")
    got = sr_gemm(dev(A), dev(B), M, N, K, CL, 0, 0, seed=5)
    assert np.array_equal(got, oracle.chunk_gemm_sr(A, B, CL, seed=5))


def test_sr_gemm_degenerate():
    say("chunk_gemm_sr K = 0")
    A = torch.zeros((5, 1), dtype=torch.uint8, device=DEV)
    B = torch.zeros((1, 7), dtype=torch.uint8, device=DEV)
    C = torch.full((5, 7), 0x1234, dtype=torch.uint16, device=DEV)
    fp8t.chunk_gemm_sr(0, 0, 5, 7, 0, 64, A, 1, B, 7, C, 7, 1)
    assert np.all(host(C) == 0)
    # one output, K = 1
    rng = np.random.default_rng(831)
    A, B = operands(rng, 1, 1, 1, 0, 0)
    say("chunk_gemm_sr 1x1x1")
    assert np.array_equal(sr_gemm(dev(A), dev(B), 1, 1, 1, 64, 0, 0, seed=2),
                          oracle.chunk_gemm_sr(A, B, 64, seed=2))


def test_sr_gemm_padded_leading_dims():
    rng = np.random.default_rng(832)
    M, N, K, CL = 77, 45, 300, 32
    A, B = operands(rng, M, N, K, 0, 0)
    Ap = np.zeros((M, K + 5), np.uint8); Ap[:, :K] = A
    Bp = np.zeros((K, N + 3), np.uint8); Bp[:, :N] = B
    C = torch.zeros((M, N + 1), dtype=torch.uint16, device=DEV)
    say("chunk_gemm_sr padded leading dimensions")
    fp8t.chunk_gemm_sr(0, 0, M, N, K, CL, dev(Ap), K + 5, dev(Bp), N + 3, C, N + 1, 9, 1)
    assert np.array_equal(host(C)[:, :N], oracle.chunk_gemm_sr(A, B, CL, seed=9, offset=1))
