"""Pins for the oracle's chunk-based GEMM (Sec. 2.3, Fig. 3(a)).

* integer-valued operands whose sums never leave the range where FP16 is
  exact reduce the method to an ordinary integer matrix product (numpy);
* the special cases CL = 1 and CL >= K are both the plain sequential
  FP16 sum, bit for bit (a one-term chunk is exact, a single chunk is added to
  +0 exactly);
* transposition symmetry and the four operand layouts;
* the accumulation experiment of Sec. 2.3 / Fig. 3(b): with CL = 1 the sum of
  a mean-1 vector stops at 4096 (magnitudes differ by 2^11), while chunking
  tracks the exact sum;
* the error bound of recursive summation (Higham) with unit round-off 2^-10
  applied to the two levels, which is the O(N/CL + CL) bound of Sec. 2.3.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads
from tests import helpers as H

U = 2.0 ** -10          # unit round-off of a 10-bit significand


def _q(x, scale=1.0):
    return oracle.fp8_quantize(np.ascontiguousarray(x, dtype=np.float32), scale)


def _int_operands(rng, M, N, K):
    # values in {-4..4}: all exact in FP8
    a = rng.integers(-4, 5, size=(M, K)).astype(np.float32)
    b = rng.integers(-4, 5, size=(K, N)).astype(np.float32)
    return a, b


@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
@pytest.mark.parametrize("mode", [oracle.EXACT, oracle.FAST])
def test_integer_exact_region_equals_matmul(ta, tb, mode):
    rng = np.random.default_rng(300 + 2 * ta + tb)
    M, N, K = 37, 29, 40           # |sums| <= 16 * 40 = 640 < 1024: all exact
    a, b = _int_operands(rng, M, N, K)
    A = _q(a.T if ta else a)
    B = _q(b.T if tb else b)
    C = oracle.chunk_gemm(A, B, CL=7, trans_a=ta, trans_b=tb, mode=mode)
    ref = a.astype(np.int64) @ b.astype(np.int64)
    assert np.array_equal(oracle.p16_value(C), ref.astype(np.float64))


def test_cl1_equals_clk_equals_sequential_sum():
    rng = np.random.default_rng(310)
    M, N, K = 9, 11, 300
    a = rng.standard_normal((M, K)).astype(np.float32)
    b = (rng.standard_normal((K, N)) * 3).astype(np.float32)
    A, B = _q(a), _q(b)
    c1 = oracle.chunk_gemm(A, B, CL=1)
    ck = oracle.chunk_gemm(A, B, CL=K)
    cbig = oracle.chunk_gemm(A, B, CL=10 * K)
    assert np.array_equal(c1, ck) and np.array_equal(ck, cbig)
    # sequential FP16 sum built from the addition primitive alone
    prods = oracle.mul8(A[:, :, None], B[None, :, :])       # M x K x N
    S = np.zeros((M, N), dtype=np.uint16)
    for k in range(K):
        S = oracle.add16(S, prods[:, k, :])
    assert np.array_equal(S, c1)


def test_two_level_structure_from_primitives():
    """C(i,j) for CL = 8 equals: sum each chunk sequentially in FP16, then sum
    the chunk results sequentially in FP16 (built here from add16/mul8)."""
    rng = np.random.default_rng(311)
    M, N, K, CL = 5, 6, 61, 8
    A = _q(rng.standard_normal((M, K)))
    B = _q(rng.standard_normal((K, N)) * 5)
    C = oracle.chunk_gemm(A, B, CL=CL)
    prods = oracle.mul8(A[:, :, None], B[None, :, :])
    S = np.zeros((M, N), dtype=np.uint16)
    for c0 in range(0, K, CL):
        P = np.zeros((M, N), dtype=np.uint16)
        for k in range(c0, min(K, c0 + CL)):
            P = oracle.add16(P, prods[:, k, :])
        S = oracle.add16(S, P)
    assert np.array_equal(S, C)
    # the inter-chunk order matters: reversing the chunk order changes bits
    # on data like this, so the test above does exercise the order
    assert not np.array_equal(C, oracle.chunk_gemm(A[:, ::-1], B[::-1, :], CL=CL))


def test_transposition_symmetry_and_layouts():
    rng = np.random.default_rng(312)
    M, N, K = 23, 17, 130
    a = _q(rng.standard_normal((M, K)))
    b = _q(rng.standard_normal((K, N)))
    C = oracle.chunk_gemm(a, b, CL=16)
    Ct = oracle.chunk_gemm(np.ascontiguousarray(b.T), np.ascontiguousarray(a.T), CL=16)
    assert np.array_equal(C, Ct.T)
    for ta in (0, 1):
        for tb in (0, 1):
            A = np.ascontiguousarray(a.T) if ta else a
            B = np.ascontiguousarray(b.T) if tb else b
            assert np.array_equal(oracle.chunk_gemm(A, B, CL=16, trans_a=ta, trans_b=tb), C)


def test_selection_matrix_copies_values():
    rng = np.random.default_rng(313)
    M, K = 40, 50
    A = _q(rng.standard_normal((M, K)) * 100)
    cols = rng.permutation(K)[:20]
    Bf = np.zeros((K, 20), dtype=np.float32)
    Bf[cols, np.arange(20)] = 1.0
    C = oracle.chunk_gemm(A, _q(Bf), CL=8)
    assert np.array_equal(oracle.p16_value(C), oracle.p8_value(A[:, cols]))


def test_empty_and_degenerate_shapes():
    A = np.zeros((4, 0), dtype=np.uint8)
    B = np.zeros((0, 3), dtype=np.uint8)
    C = oracle.chunk_gemm(A, B, CL=64)
    assert C.shape == (4, 3) and np.all(C == 0)                 # K = 0 -> +0
    assert oracle.chunk_gemm(np.zeros((0, 5), np.uint8), np.zeros((5, 3), np.uint8), 4).shape == (0, 3)
    # products of -0 never give a -0 result (sums start at +0)
    A = np.full((2, 9), 0x80, dtype=np.uint8)                   # -0
    B = np.full((9, 2), 0x3C, dtype=np.uint8)                   # 1.0
    assert np.all(oracle.chunk_gemm(A, B, CL=4) == 0x0000)
    with pytest.raises(ValueError):
        oracle.chunk_gemm(A, B, CL=0)


def test_specials_propagate():
    A = np.array([[0x7C, 0x3C], [0x7C, 0x00], [0x7D, 0x3C], [0x7B, 0x7B]], dtype=np.uint8)
    B = np.array([[0x3C], [0xFC]], dtype=np.uint8)          # 1, -Inf
    C = oracle.chunk_gemm(A, B, CL=1)[:, 0]
    # Inf*1 + 1*(-Inf) = NaN; Inf*1 + 0*(-Inf) = NaN (0*Inf); NaN; 57344-Inf = -Inf
    assert list(C) == [0x7F00, 0x7F00, 0x7F00, 0xFE00]


def test_points_match_full():
    rng = np.random.default_rng(314)
    M, N, K = 31, 45, 200
    A = _q(rng.standard_normal((K, M)))
    B = _q(rng.standard_normal((N, K)))
    for mode in (oracle.EXACT, oracle.FAST):
        C = oracle.chunk_gemm(A, B, CL=64, trans_a=1, trans_b=1, mode=mode)
        r = rng.integers(0, M, 50)
        c = rng.integers(0, N, 50)
        p = oracle.chunk_gemm_points(A, B, 64, r, c, trans_a=1, trans_b=1, mode=mode)
        assert np.array_equal(p, C[r, c])


def test_fig3b_accumulation_stalls_at_4096_without_chunking():
    """Sec. 2.3, Fig. 3(b): accumulating a vector from a uniform distribution
    with mean 1 and standard deviation 1 in FP16 with nearest rounding stops
    growing once the sum reaches 4096 (the addends are then below half a step,
    magnitudes differing by >= 2^11); chunks of 32 or more track the exact sum."""
    x = workloads.accumulation_vector(12000)
    a = _q(x)
    one = np.full((12000, 1), 0x3C, dtype=np.uint8)
    vals = oracle.p8_value(a)
    for L in (6000, 8000, 12000):
        A = np.ascontiguousarray(a[None, :L])
        B = np.ascontiguousarray(one[:L])
        s1 = oracle.p16_value(oracle.chunk_gemm(A, B, CL=1))[0, 0]
        sk = oracle.p16_value(oracle.chunk_gemm(A, B, CL=L))[0, 0]
        exact = float(np.sum(vals[:L]))          # exact: small dyadic values
        assert s1 == 4096.0 and sk == 4096.0
        assert exact > 1.4 * 4096 * (L / 6000)   # far above the stall
        for CL in (32, 64):
            sc = oracle.p16_value(oracle.chunk_gemm(A, B, CL=CL))[0, 0]
            assert abs(sc - exact) / exact < 0.02, (L, CL, sc, exact)
    # the stall value is absorbing: every addend is lost at 4096
    s = oracle.rn16(4096.0)[()]
    assert vals.max() < 4 and vals.min() > -2
    for v in np.unique(a):
        assert oracle.add16(s, oracle.mul8(v, 0x3C))[()] == s


@pytest.mark.parametrize("CL", [1, 8, 64, 256, 4096])
def test_error_bound_two_level_recursive_summation(CL):
    """|C - sum_k a_k b_k| <= ((CL - 1) + (ceil(K/CL) - 1)) * u * sum |a_k b_k|
    * (1 + u)^2, u = 2^-10: Higham's bound for recursive summation applied to the
    intra-chunk sums and to the sum of the chunk sums (Sec. 2.3 quotes the
    O(N/CL + CL) order)."""
    K = 4096
    A32, B32 = workloads.sweep_gemm(K, M=8, N=8)
    A, B = _q(A32), _q(B32)
    va, vb = oracle.p8_value(A), oracle.p8_value(B)
    C = oracle.p16_value(oracle.chunk_gemm(A, B, CL=CL, trans_a=1))
    exact = va.T @ vb                         # error of float64 here is < 1e-12 rel
    absum = np.abs(va).T @ np.abs(vb)
    nch = -(-K // CL)
    bound = ((min(CL, K) - 1) + (nch - 1)) * U * absum * (1 + U) ** 2
    assert np.all(np.abs(C - exact) <= bound + 1e-9 * absum)


def test_chunking_reduces_error_on_long_sums():
    """Sec. 4.2: chunk sizes in the middle range beat both extremes (no
    chunking, or one chunk) on long weight-gradient-like sums."""
    K = 4096
    A32, B32 = workloads.sweep_gemm(K, M=16, N=16)
    A, B = _q(A32), _q(B32)
    exact = oracle.p8_value(A).T @ oracle.p8_value(B)
    err = {}
    for CL in (1, 64, K):
        C = oracle.p16_value(oracle.chunk_gemm(A, B, CL=CL, trans_a=1))
        err[CL] = np.linalg.norm(C - exact) / np.linalg.norm(exact)
    assert err[64] < 0.5 * err[1] and err[1] == err[K]


def test_fast_mode_rounds_each_chunk_once():
    rng = np.random.default_rng(315)
    M, N, K, CL = 6, 7, 150, 32
    A = _q(rng.standard_normal((M, K)))
    B = _q(rng.standard_normal((K, N)) * 7)
    C = oracle.chunk_gemm(A, B, CL=CL, mode=oracle.FAST)
    va, vb = oracle.p8_value(A), oracle.p8_value(B)
    ref = np.zeros((M, N), dtype=np.uint16)
    for i in range(M):
        for j in range(N):
            S = 0
            for c0 in range(0, K, CL):
                exact = sum(Fraction(float(va[i, k])) * Fraction(float(vb[k, j]))
                            for k in range(c0, min(K, c0 + CL)))
                P = H.brute_rn16(exact) if exact != 0 else 0
                S = int(oracle.add16(S, P))
            ref[i, j] = S
    assert np.array_equal(C, ref)
    # one-term chunks are exact in both modes
    assert np.array_equal(oracle.chunk_gemm(A, B, CL=1, mode=oracle.FAST),
                          oracle.chunk_gemm(A, B, CL=1))
