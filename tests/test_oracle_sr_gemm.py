"""Pins for the oracle's chunk-based GEMM with stochastic rounding after every
P16 addition (Sec. 2.3: the two rounding modes after FP16 additions;
Fig. 3(b): stochastic rounding follows the FP32 sum where nearest rounding
stalls).

* where every sum is exact in P16 the rounding mode cannot matter: the result
  is the ordinary integer matrix product, for any seed;
* one rounding with a known discarded fraction rounds up with exactly that
  probability (checked over 4096 independent outputs, for the intra-chunk and
  the inter-chunk additions separately), and only to the two neighbours;
* the accumulation experiment of Fig. 3(b) without chunking: nearest
  rounding stops at 4096, stochastic rounding stays close to the exact sum;
* an independent formulation -- numpy float32 additions and rational
  arithmetic for Eq. (1) -- reproduces the oracle bit for bit on small cases.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads


def _q(x, scale=1.0):
    return oracle.fp8_quantize(np.ascontiguousarray(x, dtype=np.float32), scale)


@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_sr_exact_region_equals_matmul(ta, tb):
    rng = np.random.default_rng(900 + 2 * ta + tb)
    M, N, K = 9, 7, 40                      # |sums| <= 640 < 1024: exact in P16
    a = rng.integers(-4, 5, size=(M, K)).astype(np.float32)
    b = rng.integers(-4, 5, size=(K, N)).astype(np.float32)
    A = _q(a.T if ta else a)
    B = _q(b.T if tb else b)
    want = oracle.fp16_quantize((a.astype(np.int64) @ b.astype(np.int64)).astype(np.float32))
    for CL in (1, 3, 16, 64):
        for seed in (0, 1, 2 ** 40 + 3):
            got = oracle.chunk_gemm_sr(A, B, CL, ta, tb, seed=seed, offset=CL)
            assert np.array_equal(got, want), (CL, seed)


@pytest.mark.parametrize("CL", [1, 2])
def test_sr_single_rounding_probability(CL):
    """1 + 3 * 2^-11 lies 3/4 of a P16 step (2^-9) above 1: it must become
    1 + 2^-9 with probability exactly 3/4 (F = 49152 of 65536 uniforms).  With
    CL = 2 that rounding is the intra-chunk addition of product 1, with CL = 1
    the inter-chunk addition of chunk 1."""
    M = 4096
    A = np.zeros((M, 2), np.uint8)
    A[:, 0] = _q(np.float32(1.0))
    A[:, 1] = _q(np.float32(3 * 2.0 ** -11))
    assert oracle.p8_value(A[0, 1]) == 3 * 2.0 ** -11
    B = np.full((2, 1), _q(np.float32(1.0)), np.uint8)
    for seed, offset in ((5, 0), (6, 9)):
        v = oracle.p16_value(oracle.chunk_gemm_sr(A, B, CL, seed=seed, offset=offset))[:, 0]
        assert set(np.unique(v)) <= {1.0, 1.0 + 2.0 ** -9}
        frac_up = float(np.mean(v > 1.0))
        sigma = math.sqrt(0.75 * 0.25 / M)
        assert abs(frac_up - 0.75) < 5 * sigma, (seed, frac_up)
    # nearest rounding would always round up (3/4 > 1/2)
    assert np.all(oracle.p16_value(oracle.chunk_gemm(A, B, CL)) == 1.0 + 2.0 ** -9)


def test_fig3b_stochastic_rounding_follows_exact_sum():
    """Fig. 3(b): with nearest rounding and no chunking the sum of the mean-1
    vector stalls at 4096; with stochastic rounding it follows the exact sum
    (unbiased; the spread is that of the rounding noise)."""
    L, R = 12000, 32
    x = workloads.accumulation_vector(L)
    a = _q(x)
    exact = float(np.sum(oracle.p8_value(a)))
    A = np.ascontiguousarray(np.broadcast_to(a[None, :], (R, L)))
    B = np.full((L, 1), 0x3C, np.uint8)
    assert oracle.p16_value(oracle.chunk_gemm(A[:1], B, CL=L))[0, 0] == 4096.0
    s = oracle.p16_value(oracle.chunk_gemm_sr(A, B, L, seed=21))[:, 0]
    assert len(np.unique(s)) > 1                       # rows draw different bits
    assert abs(float(np.mean(s)) - exact) / exact < 0.02, (float(np.mean(s)), exact)
    assert np.all(np.abs(s - exact) / exact < 0.2)


def _sr_rational(x32, u):
    """Eq. (1) on the FP32 value x32 in exact rational arithmetic."""
    if np.isnan(x32):
        return float("nan")
    if np.isinf(x32):
        return float(x32)
    a = Fraction(float(abs(x32)))
    if a == 0:
        return float(x32)
    e = math.floor(math.log2(a))
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    q = Fraction(2) ** -39 if a < Fraction(2) ** -30 else Fraction(2) ** (e - 9)
    t = a / q
    n = math.floor(t)
    F = math.floor((t - n) * 65536)
    r = (n + (1 if u < F else 0)) * q
    r = float("inf") if r >= 2 ** 32 else float(r)
    return math.copysign(r, float(x32))


def _uniform(i, j, q, w3, idx, seed):
    words = oracle.philox4x32_10([i, j, q, w3], [seed & 0xFFFFFFFF, seed >> 32])
    w = int(words[idx // 2])
    return (w >> 16) if idx % 2 else (w & 0xFFFF)


@pytest.mark.parametrize("ta,tb", [(0, 0), (1, 1)])
def test_sr_independent_formulation(ta, tb):
    rng = np.random.default_rng(910 + ta)
    M, N, K, CL, seed, offset = 3, 11, 19, 4, 77, 5
    a = (rng.standard_normal((M, K)) * 8).astype(np.float32)
    b = (rng.standard_normal((K, N)) * 8).astype(np.float32)
    A, B = _q(a.T if ta else a), _q(b.T if tb else b)
    av = oracle.p8_value(A.T if ta else A)
    bv = oracle.p8_value(B.T if tb else B)
    got = oracle.p16_value(oracle.chunk_gemm_sr(A, B, CL, ta, tb, seed=seed, offset=offset))
    for i in range(M):
        for j in range(N):
            S = 0.0
            for c, c0 in enumerate(range(0, K, CL)):
                P = 0.0
                for k in range(c0, min(K, c0 + CL)):
                    x = np.float32(P) + np.float32(av[i, k] * bv[k, j])
                    P = _sr_rational(x, _uniform(i, j // 4, k // 2, 2 * offset,
                                                 4 * (k % 2) + j % 4, seed))
                x = np.float32(S) + np.float32(P)
                S = _sr_rational(x, _uniform(i, j // 8, c, 2 * offset + 1, j % 8, seed))
            assert got[i, j] == S, (i, j, got[i, j], S)
    # and it differs from nearest rounding somewhere (the roundings are live)
    rn = oracle.p16_value(oracle.chunk_gemm(A, B, CL, ta, tb))
    assert not np.array_equal(rn, got)


def test_sr_argument_checks():
    A = np.zeros((2, 3), np.uint8)
    B = np.zeros((3, 2), np.uint8)
    with pytest.raises(ValueError):
        oracle.chunk_gemm_sr(A, B, 0, seed=1)
    with pytest.raises(ValueError):
        oracle.chunk_gemm_sr(A, B, 4, seed=1, offset=2 ** 31)
    assert np.all(oracle.chunk_gemm_sr(A[:, :0], B[:0], 4, seed=1) == 0)


def _header_text():
    import os
    import re
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                        "include", "fp8train.h")
    with open(path) as f:
        text = f.read()
    text = re.sub(r"\n\s*\*\s?", " ", text)          # join comment lines
    return re.sub(r"\s+", " ", text)


def test_header_documents_the_keying_tested_above():
    """The public header states the random-bit keying that the independent
    formulation above recomputes, so a caller reproducing a call from the
    header gets the oracle's bits."""
    doc = _header_text()
    seg = doc[doc.index("chunk_gemm_sr -- "):doc.index("int chunk_gemm_sr(")]
    for phrase in ("key = (seed low, seed high)",
                   "low half first: uniform q is half q mod 2 of word q / 2",
                   "uniform 4 (k mod 2) + (j mod 4) of the block with counter "
                   "(i, j / 4, k / 2, 2 * offset)",
                   "uniform j mod 8 of the block with counter (i, j / 8, c, 2 * offset + 1)"):
        assert phrase in seg, phrase
