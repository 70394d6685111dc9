"""GPU parity of chunk_gemm_p16 (FP16 operands, products rounded to FP16,
chunk-based FP16 accumulation) with the oracle, bit for bit: every layout,
ragged chunks, CL = 1 and CL >= K, whole and shared-out tiles, subnormal and
overflowing products, specials, K = 0, and the last layer of the speech DNN
(256 x 6000 x 1024 and its backward GEMMs) on one output per 16 x 16 block."""
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


def p16(x):
    return oracle.fp16_quantize(np.asarray(x, np.float32))


def gemm16(A, B, M, N, K, CL, ta, tb, use_ws=True):
    wb = fp8t.chunk_gemm_p16_workspace_size(ta, tb, M, N, K, CL) if use_ws else 0
    ws = torch.empty(wb, dtype=torch.uint8, device=DEV) if wb else None
    C = torch.full((M, N), 0xABCD, dtype=torch.uint16, device=DEV)
    fp8t.chunk_gemm_p16(ta, tb, M, N, K, CL, A, A.shape[-1], B, B.shape[-1], C, N, ws, wb)
    return host(C)


SHAPES = [(130, 67, 333, 64), (64, 96, 1000, 7), (33, 47, 700, 700), (70, 150, 600, 1),
          (5, 3, 17, 4), (128, 64, 2048, 64)]


@pytest.mark.parametrize("guard", ["1", "0"])
@pytest.mark.parametrize("plan", ["auto", "shared", "no_ws"])
@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_p16_gemm_matches_oracle(ta, tb, plan, guard, monkeypatch):
    monkeypatch.setenv("FP8T_GEMM_GUARD", guard)
    if plan == "shared":
        monkeypatch.setenv("FP8T_GEMM_SPLIT", "1")
        monkeypatch.setenv("FP8T_GEMM_WGS", "7")
    rng = np.random.default_rng(980 + 2 * ta + tb)
    for (M, N, K, CL) in SHAPES:
        a = rng.standard_normal((M, K)) * 2.0
        b = rng.standard_normal((K, N)) * 0.5
        a[rng.random(a.shape) < 0.03] = 0.0
        A, B = p16(a.T if ta else a), p16(b.T if tb else b)
        say(f"chunk_gemm_p16 plan={plan} guard={guard} ta={ta} tb={tb} {M}x{N}x{K} CL={CL}")
        got = gemm16(dev(A), dev(B), M, N, K, CL, ta, tb, use_ws=plan != "no_ws")
        ref = oracle.chunk_gemm_p16(A, B, CL, ta, tb)
        assert np.array_equal(got, ref), (M, N, K, CL, np.argwhere(got != ref)[:5])


@pytest.mark.parametrize("guard", ["1", "0"])
def test_p16_gemm_ranges_and_specials(guard, monkeypatch):
    """Operands whose products leave the guarded path's range (overflowing
    products, Inf, NaN): the pieces fall back and must still match; with
    guard 0 every piece runs on the 2^96-domain path."""
    monkeypatch.setenv("FP8T_GEMM_GUARD", guard)
    rng = np.random.default_rng(985)
    M, N, K, CL = 70, 40, 256, 64
    # magnitudes from 2^-39 to 2^31: subnormal and overflowing products
    a = np.exp2(rng.uniform(-39, 31, (M, K))) * np.sign(rng.standard_normal((M, K)))
    b = np.exp2(rng.uniform(-20, 5, (K, N))) * np.sign(rng.standard_normal((K, N)))
    A, B = p16(a), p16(b)
    A[3, 5] = 0x7E00                      # +Inf
    A[4, 6] = 0x7F00                      # NaN
    A[5, :] = 0x0001                      # smallest subnormal
    A[6, :] = 0x7DFF                      # largest finite
    say("chunk_gemm_p16 ranges and specials")
    got = gemm16(dev(A), dev(B), M, N, K, CL, 0, 0)
    assert np.array_equal(got, oracle.chunk_gemm_p16(A, B, CL))


@pytest.mark.parametrize("guard", ["1", "0"])
def test_p16_gemm_small_magnitudes(guard, monkeypatch):
    """Magnitudes from 2^-39 to 2^-5 times 2^-20 to 1: most products lie in
    FP16's subnormal range or underflow to 0, every piece passes the guard."""
    monkeypatch.setenv("FP8T_GEMM_GUARD", guard)
    rng = np.random.default_rng(986)
    M, N, K, CL = 90, 70, 300, 32
    a = np.exp2(rng.uniform(-39, -5, (M, K))) * np.sign(rng.standard_normal((M, K)))
    b = np.exp2(rng.uniform(-20, 0, (K, N))) * np.sign(rng.standard_normal((K, N)))
    A, B = p16(a), p16(b)
    say(f"chunk_gemm_p16 small magnitudes guard={guard}")
    got = gemm16(dev(A), dev(B), M, N, K, CL, 0, 0)
    assert np.array_equal(got, oracle.chunk_gemm_p16(A, B, CL))


@pytest.mark.parametrize("row_scale", [2.0 ** -28, 2.0 ** 17])
def test_p16_gemm_guard_rows(row_scale, monkeypatch):
    """One row of A scaled among ordinary ones.  2^-28: products in FP16's
    subnormal range, rounded on the guarded path itself.  2^17: only the
    tiles holding the row fail the overflow bound (shared plan: only their
    pieces) and are recomputed in the 2^96 domain."""
    monkeypatch.setenv("FP8T_GEMM_SPLIT", "1")
    monkeypatch.setenv("FP8T_GEMM_WGS", "9")
    rng = np.random.default_rng(987)
    M, N, K, CL = 200, 130, 700, 64
    A = p16(rng.standard_normal((M, K)))
    B = p16(rng.standard_normal((K, N)))
    A[150, :] = p16(rng.standard_normal(K) * row_scale)
    say(f"chunk_gemm_p16 guard rows scale={row_scale}")
    got = gemm16(dev(A), dev(B), M, N, K, CL, 0, 0)
    assert np.array_equal(got, oracle.chunk_gemm_p16(A, B, CL))


def test_p16_gemm_empty_k():
    say("chunk_gemm_p16 K = 0")
    A = torch.zeros((5, 1), dtype=torch.uint16, device=DEV)
    B = torch.zeros((1, 7), dtype=torch.uint16, device=DEV)
    C = torch.full((5, 7), 0x1234, dtype=torch.uint16, device=DEV)
    fp8t.chunk_gemm_p16(0, 0, 5, 7, 0, 64, A, 1, B, 7, C, 7)
    assert np.all(host(C) == 0)


def test_p16_gemm_last_layer_shapes(monkeypatch):
    """The speech DNN's last layer (1024 -> 6000, batch 256): Forward,
    Backward (trans_b) and Gradient (trans_a) GEMMs in the plan the benchmark
    runs (workspace from the query), one output in every 16 x 16 block of C
    -- the smallest workgroup tile, so every tile and every shared tile's
    pieces are checked -- plus the corners; for the two GEMMs with tiles
    shared out, also with the guard off (the 2^96 path throughout)."""
    from tests.test_gpu_workloads import tile_points
    rng = np.random.default_rng(986)
    X = p16(np.maximum(rng.standard_normal((256, 1024)), 0))
    W = p16(rng.standard_normal((1024, 6000)) / 32.0)
    E = p16(rng.standard_normal((256, 6000)) * 1e-3 * 1000)
    Xd, Wd, Ed = dev(X), dev(W), dev(E)
    for (A, B, Ad, Bd, M, N, K, ta, tb, what) in (
            (X, W, Xd, Wd, 256, 6000, 1024, 0, 0, "fwd"),
            (E, W, Ed, Wd, 256, 1024, 6000, 0, 1, "dgrad"),
            (X, E, Xd, Ed, 1024, 6000, 256, 1, 0, "wgrad")):
        r, c = tile_points(M, N, 990 + ta + 2 * tb, block=16, per=1)
        say(f"chunk_gemm_p16 last layer {what} {M}x{N}x{K}: {r.size} outputs checked")
        ref = oracle.chunk_gemm_p16_points(A, B, 64, r, c, ta, tb)
        got = gemm16(Ad, Bd, M, N, K, 64, ta, tb)
        assert np.array_equal(got[r, c], ref), (what, np.flatnonzero(got[r, c] != ref)[:5])
        if fp8t.chunk_gemm_p16_workspace_size(ta, tb, M, N, K, 64) > 0:
            monkeypatch.setenv("FP8T_GEMM_GUARD", "0")
            say(f"chunk_gemm_p16 last layer {what}, guard off")
            got = gemm16(Ad, Bd, M, N, K, 64, ta, tb)
            monkeypatch.delenv("FP8T_GEMM_GUARD")
            assert np.array_equal(got[r, c], ref), (what, np.flatnonzero(got[r, c] != ref)[:5])
