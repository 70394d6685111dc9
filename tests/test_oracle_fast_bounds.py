"""Pins for the bounds on the fast mode's results (the FP32 chunk sums of the
build's fast mode, then the paper's FP16 rounding and inter-chunk chain of
Sec. 2.3).

* the fast oracle (exact chunk sums) always lies inside the bounds, and with
  one product per chunk the bounds collapse onto the exact-mode result;
* FP32 sums of every chunk taken in several orders -- sequential, reversed,
  pairwise, largest magnitude first, random permutations -- then rounded and
  chained with the oracle's FP16 addition, always lie inside the bounds (also
  on data built to make FP32 order matter);
* the bounds are tight enough to reject the failures a tolerance in units of
  sum|p| lets through: an all-zero result, the last chunk dropped, a middle
  chunk dropped, chunks shifted by one product.
"""
import numpy as np
import pytest

import oracle
from tests.helpers import within_fast_bounds

RNG = np.random.default_rng(1200)


def _operands(rng, M, N, K, spread=1.0):
    a = (rng.standard_normal((M, K)) * spread).astype(np.float32)
    b = rng.standard_normal((K, N)).astype(np.float32)
    a[rng.random(a.shape) < 0.05] = 0.0
    b[rng.random(b.shape) < 0.02] *= 64.0
    return oracle.fp8_quantize(a), oracle.fp8_quantize(b)


def fp32_chunked(A, B, CL, order, rng):
    """The fast mode's arithmetic simulated on the CPU: each chunk's products
    (exact in float32) summed in float32 in the given order, rounded to FP16,
    then the FP16 chain of chunk sums."""
    va, vb = oracle.p8_value(A).astype(np.float32), oracle.p8_value(B).astype(np.float32)
    M, K = va.shape
    N = vb.shape[1]
    C = np.zeros((M, N), np.uint16)
    for i in range(M):
        for j in range(N):
            p = (va[i, :] * vb[:, j]).astype(np.float32)
            S = np.uint16(0)
            for c0 in range(0, K, CL):
                q = p[c0:c0 + CL]
                if order == "reverse":
                    q = q[::-1]
                elif order == "bigfirst":
                    q = q[np.argsort(-np.abs(q), kind="stable")]
                elif order == "random":
                    q = q[rng.permutation(q.size)]
                if order == "pairwise":
                    s = np.add.reduce(q, dtype=np.float32)   # numpy: pairwise blocks
                else:
                    s = np.float32(0.0)
                    for t in q:
                        s = np.float32(s + t)
                P = oracle.rn16(np.float64(s))
                S = oracle.add16(S, P)
            C[i, j] = S
    return C


@pytest.mark.parametrize("M,N,K,CL", [(7, 5, 300, 64), (6, 4, 333, 16), (5, 5, 200, 200),
                                      (4, 6, 129, 1)])
def test_fast_oracle_and_fp32_orders_inside_bounds(M, N, K, CL):
    A, B = _operands(RNG, M, N, K)
    lo, hi = oracle.chunk_gemm_fast_bounds(A, B, CL)
    assert within_fast_bounds(oracle.chunk_gemm(A, B, CL, mode=oracle.FAST), lo, hi).all()
    if CL == 1:
        assert np.array_equal(lo, hi)
        assert np.array_equal(lo, oracle.chunk_gemm(A, B, 1))
    rng = np.random.default_rng(1201)
    for order in ("sequential", "reverse", "pairwise", "bigfirst", "random", "random"):
        C = fp32_chunked(A, B, CL, order, rng)
        assert within_fast_bounds(C, lo, hi).all(), order


def test_fp32_order_sensitive_data_inside_bounds():
    """Chunks mixing products of very different sizes and signs, where the
    float32 result depends on the order."""
    rng = np.random.default_rng(1202)
    M, N, K, CL = 6, 6, 256, 64
    # every chunk opens with +X and -X (X = 1.25 * 2^22) and continues with
    # small products: summed in order, the small ones are absorbed while X is
    # in the sum; largest first, X cancels exactly and they all count
    a = (rng.standard_normal((M, K)) * 0.125).astype(np.float32)
    b = rng.standard_normal((K, N)).astype(np.float32)
    a[:, 0::CL] = 2560.0
    a[:, 1::CL] = -2560.0
    b[0::CL, :] = 2048.0
    b[1::CL, :] = 2048.0
    A, B = oracle.fp8_quantize(a), oracle.fp8_quantize(b)
    lo, hi = oracle.chunk_gemm_fast_bounds(A, B, CL)
    seen = set()
    for order in ("sequential", "reverse", "pairwise", "bigfirst", "random", "random", "random"):
        C = fp32_chunked(A, B, CL, order, rng)
        assert within_fast_bounds(C, lo, hi).all(), order
        seen.add(C.tobytes())
    assert len(seen) > 1            # the order mattered on this data
    assert (lo != hi).any()


@pytest.mark.parametrize("M,N,K,CL", [(130, 67, 333, 64), (37, 29, 100, 16), (19, 23, 1030, 256),
                                      (33, 47, 400, 48), (64, 64, 2304, 64)])
def test_bounds_reject_plausible_failures(M, N, K, CL):
    A, B = _operands(RNG, M, N, K)
    lo, hi = oracle.chunk_gemm_fast_bounds(A, B, CL)
    ok = oracle.chunk_gemm(A, B, CL, mode=oracle.FAST)
    assert within_fast_bounds(ok, lo, hi).all()
    single = float(np.mean(lo == hi))
    assert single > 0.3, single
    last = (K - 1) // CL * CL                    # start of the last chunk
    mid = (K // CL // 2) * CL
    mutants = {
        "zero": np.zeros_like(ok),
        "last chunk dropped": oracle.chunk_gemm(A[:, :last], B[:last, :], CL, mode=oracle.FAST)
        if last > 0 else np.zeros_like(ok),
        "middle chunk dropped": oracle.chunk_gemm(
            np.concatenate([A[:, :mid], A[:, mid + CL:]], 1),
            np.concatenate([B[:mid, :], B[mid + CL:, :]], 0), CL, mode=oracle.FAST),
        "chunks shifted by one": oracle.chunk_gemm(
            np.concatenate([np.zeros((M, 1), np.uint8), A], 1),
            np.concatenate([np.zeros((1, N), np.uint8), B], 0), CL, mode=oracle.FAST),
    }
    for name, C in mutants.items():
        if name == "middle chunk dropped" and K < 3 * CL:
            continue
        bad = 1.0 - float(np.mean(within_fast_bounds(C, lo, hi)))
        assert bad > 0.3, (name, bad)
