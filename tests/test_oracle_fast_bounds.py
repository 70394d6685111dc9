"""Pins for the bounds on the fast mode's results (chunk sums formed without
per-addition FP16 rounding, then the paper's FP16 rounding and inter-chunk
chain of Sec. 2.3).

Chunk sums in FP32 on the vector ALUs (matrix_core=False):
* the fast oracle (exact chunk sums) always lies inside the bounds, and with
  one product per chunk the bounds collapse onto the exact-mode result;
* FP32 sums of every chunk taken in several orders -- sequential, reversed,
  pairwise, largest magnitude first, random permutations -- then rounded and
  chained with the oracle's FP16 addition, always lie inside the bounds (also
  on data built to make FP32 order matter).
Chunk sums on the FP8 matrix cores (matrix_core=True):
* a simulation of the measured arithmetic written here (groups of 8 products
  truncated to 2^(E-13) of the group's largest exponent sum, the group sums
  combined in float32 in several orders) lies inside the bounds;
* a chunk built so that the truncation moves its sum across an FP16 rounding
  point gets single-valued bounds on the truncated side, excluding the exact
  sum's rounding.
Both:
* the bounds are tight enough to reject the failures a tolerance in units of
  sum|p| lets through: an all-zero result, the last chunk dropped, a middle
  chunk dropped, chunks shifted by one product.
"""
from fractions import Fraction

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
    lo, hi = oracle.chunk_gemm_fast_bounds(A, B, CL, matrix_core=False)
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
    lo, hi = oracle.chunk_gemm_fast_bounds(A, B, CL, matrix_core=False)
    seen = set()
    for order in ("sequential", "reverse", "pairwise", "bigfirst", "random", "random", "random"):
        C = fp32_chunked(A, B, CL, order, rng)
        assert within_fast_bounds(C, lo, hi).all(), order
        seen.add(C.tobytes())
    assert len(seen) > 1            # the order mattered on this data
    assert (lo != hi).any()


def _p8_exponent(c):
    e = (int(c) >> 2) & 31
    return -14 if e == 0 else e - 15


def matrix_core_chunked(A, B, CL, order, rng):
    """The measured arithmetic of the FP8 matrix cores, simulated: each
    aligned group of 8 products truncated towards zero to a multiple of
    2^(E - 13), E the largest e_a + e_b of its non-zero products; the group
    sums added in float32 in the given order; then FP16 rounding and chain."""
    va, vb = oracle.p8_value(A), oracle.p8_value(B)
    M, K = A.shape
    N = B.shape[1]
    C = np.zeros((M, N), np.uint16)
    for i in range(M):
        for j in range(N):
            S = np.uint16(0)
            for c0 in range(0, K, CL):
                groups = []
                for g0 in range(c0, min(K, c0 + CL), 8):
                    ks = range(g0, min(K, g0 + 8, c0 + CL))
                    ps = [(Fraction(float(va[i, k])) * Fraction(float(vb[k, j])),
                           _p8_exponent(A[i, k]) + _p8_exponent(B[k, j])) for k in ks]
                    nz = [e for p, e in ps if p != 0]
                    if not nz:
                        continue
                    q = Fraction(2) ** (max(nz) - 13)
                    tot = Fraction(0)
                    for p, _ in ps:
                        t = abs(p) // q * q
                        tot += t if p >= 0 else -t
                    groups.append(np.float32(float(tot)))   # exact: <= 19 significant bits
                if order == "reverse":
                    groups = groups[::-1]
                elif order == "random":
                    groups = [groups[x] for x in rng.permutation(len(groups))]
                s = np.float32(0.0)
                for g in groups:
                    s = np.float32(s + g)
                S = oracle.add16(S, oracle.rn16(np.float64(s)))
            C[i, j] = S
    return C


@pytest.mark.parametrize("M,N,K,CL", [(6, 5, 300, 64), (5, 6, 333, 16), (4, 4, 160, 160)])
def test_matrix_core_simulation_inside_bounds(M, N, K, CL):
    A, B = _operands(RNG, M, N, K)
    lo, hi = oracle.chunk_gemm_fast_bounds(A, B, CL, matrix_core=True)
    rng = np.random.default_rng(1203)
    for order in ("sequential", "reverse", "random"):
        C = matrix_core_chunked(A, B, CL, order, rng)
        assert within_fast_bounds(C, lo, hi).all(), order


def test_matrix_core_truncation_decides_the_rounding():
    """One chunk of 16: 256 and fifteen products 0.0546875 (= 2^-5 + 2^-6 +
    2^-7, below the grid 2^(8 - 13) = 2^-5 of the group holding 256, in
    the first group, and exactly representable in the second).  Exact sum
    256.8203125 -> FP16 257; the matrix core's sum 256 + 7 * 2^-5 +
    8 * 0.0546875 = 256.65625 -> FP16 256.5."""
    A = oracle.fp8_quantize(np.float32([[256.0] + [0.0546875] * 15]))
    B = oracle.fp8_quantize(np.ones((16, 1), np.float32))
    assert oracle.p8_value(A[0, 1]) == 0.0546875
    lo, hi = oracle.chunk_gemm_fast_bounds(A, B, 16, matrix_core=True)
    assert lo[0, 0] == hi[0, 0]
    assert oracle.p16_value(lo[0, 0]) == 256.5
    assert oracle.p16_value(oracle.chunk_gemm(A, B, 16, mode=oracle.FAST)[0, 0]) == 257.0
    # the vector-ALU bounds admit only the exact sum's rounding
    lo2, hi2 = oracle.chunk_gemm_fast_bounds(A, B, 16, matrix_core=False)
    assert oracle.p16_value(lo2[0, 0]) == oracle.p16_value(hi2[0, 0]) == 257.0


@pytest.mark.parametrize("mc", [False, True])
@pytest.mark.parametrize("M,N,K,CL", [(130, 67, 333, 64), (37, 29, 100, 16), (19, 23, 1030, 256),
                                      (33, 47, 400, 48), (64, 64, 2304, 64)])
def test_bounds_reject_plausible_failures(M, N, K, CL, mc):
    A, B = _operands(RNG, M, N, K)
    lo, hi = oracle.chunk_gemm_fast_bounds(A, B, CL, matrix_core=mc)
    ok = oracle.chunk_gemm(A, B, CL, mode=oracle.FAST)
    if not mc:
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
