"""Pins for the oracle's GEMM with FP16 operands (Sec. 3: the last layer's
GEMMs stay in FP16; read as Fig. 3(a) with FP_mult = FP_acc = FP16):

* integer operands whose sums stay where FP16 is exact reduce it to the
  integer matrix product, for every layout and chunk length;
* each product is rounded to FP16 before it is added: found by search, a case
  where rounding the product first changes the sum (a tie created by the
  product's rounding) must follow the rounded product;
* products below 2^-30 land on the subnormal grid (step 2^-39, ties to even);
* CL = 1 and CL >= K are both the plain sequential FP16 sum of the rounded
  products, bit for bit;
* transposition symmetry;
* recursive-summation error bound (Higham), one extra rounding per product.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle

U = 2.0 ** -10


def p16(x):
    return oracle.fp16_quantize(np.asarray(x, np.float32))


def rn16_frac(x):
    """Nearest FP16 value of a non-zero rational in the normal range, ties to
    even (an independent formulation for the search below)."""
    s = -1 if x < 0 else 1
    a = abs(x)
    e = math.floor(math.log2(a))
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    q = Fraction(2) ** (e - 9)
    t = a / q
    n = math.floor(t)
    r = t - n
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return s * n * q


@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_integer_region_equals_matmul(ta, tb):
    rng = np.random.default_rng(970 + 2 * ta + tb)
    M, N, K = 7, 9, 16
    a = rng.integers(-8, 9, size=(M, K))
    b = rng.integers(-8, 9, size=(K, N))
    A = p16((a.T if ta else a).astype(np.float32))
    B = p16((b.T if tb else b).astype(np.float32))
    want = p16((a @ b).astype(np.float32))
    for CL in (1, 3, 16, 100):
        assert np.array_equal(oracle.chunk_gemm_p16(A, B, CL, ta, tb), want)


def test_products_are_rounded_before_the_addition():
    """P = 1 + 2^-9, then a1 b1 = 778 x 1011 x 2^-28 (found by a search over
    significands): rounding the product to FP16 first moves the sum across a
    rounding boundary."""
    P = Fraction(513, 512)
    a1, b1 = Fraction(778, 512), Fraction(1011, 512) * Fraction(1, 2 ** 10)
    assert rn16_frac(P + rn16_frac(a1 * b1)) != rn16_frac(P + a1 * b1)
    A = p16(np.float32([[float(P), float(a1)]]))
    B = p16(np.float32([[1.0], [float(b1)]]))
    assert oracle.p16_value(A)[0, 1] == float(a1) and oracle.p16_value(B)[1, 0] == float(b1)
    got = oracle.p16_value(oracle.chunk_gemm_p16(A, B, 64))[0, 0]
    assert got == float(rn16_frac(P + rn16_frac(a1 * b1)))


def test_subnormal_products():
    for a, want in ((2.0 ** -20, 0.0),                        # 2^-40: tie -> even (0)
                    (2.0 ** -20 * (1 + 2.0 ** -9), 2.0 ** -39),
                    (2.0 ** -19 * 1.5, 2.0 ** -39 * 4)):      # 4.5 x 2^-39: tie -> 4
        A = p16(np.float32([[a]]))
        B = p16(np.float32([[a]]))
        assert oracle.p16_value(oracle.chunk_gemm_p16(A, B, 1))[0, 0] == want, a


def test_cl1_equals_one_chunk():
    rng = np.random.default_rng(971)
    A = p16(rng.standard_normal((6, 300)) * 3)
    B = p16(rng.standard_normal((300, 5)) * 3)
    c1 = oracle.chunk_gemm_p16(A, B, 1)
    assert np.array_equal(c1, oracle.chunk_gemm_p16(A, B, 300))
    assert np.array_equal(c1, oracle.chunk_gemm_p16(A, B, 10 ** 6))
    assert not np.array_equal(c1, oracle.chunk_gemm_p16(A, B, 16))


def test_transposition_and_layouts():
    rng = np.random.default_rng(972)
    A = p16(rng.standard_normal((11, 70)))
    B = p16(rng.standard_normal((70, 13)))
    C = oracle.chunk_gemm_p16(A, B, 8)
    assert np.array_equal(C, oracle.chunk_gemm_p16(A.T.copy(), B, 8, 1, 0))
    assert np.array_equal(C, oracle.chunk_gemm_p16(A, B.T.copy(), 8, 0, 1))
    assert np.array_equal(C.T, oracle.chunk_gemm_p16(B.T.copy(), A.T.copy(), 8))


def test_error_bound():
    rng = np.random.default_rng(973)
    K = 2000
    A = p16(rng.standard_normal((16, K)))
    B = p16(rng.standard_normal((K, 12)))
    av, bv = oracle.p16_value(A), oracle.p16_value(B)
    exact = av @ bv
    absum = np.abs(av) @ np.abs(bv)
    for CL in (1, 16, 64, K):
        nch = -(-K // CL)
        got = oracle.p16_value(oracle.chunk_gemm_p16(A, B, CL))
        bound = (1 + (min(CL, K) - 1) + (nch - 1)) * U * (1 + U) ** 2 * absum
        assert np.all(np.abs(got - exact) <= bound), CL
