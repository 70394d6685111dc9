"""Pins for the oracle's FP16 addition with round-to-nearest (Sec. 2.2, 2.3).

* brute-force nearest-neighbour search over all 65536 FP16 codes, with the
  exact sum formed from rationals (a different algorithm from the oracle's);
* the swamping threshold of Sec. 2.3: an addend is lost entirely once the
  magnitudes differ by more than 2^(mantissa+1) = 2^10;
* algebraic invariants of correctly rounded addition.
"""
from fractions import Fraction

import numpy as np

import oracle
from tests import helpers as H


def _brute_add(ca, cb):
    a, b = H.to_fraction16(ca), H.to_fraction16(cb)
    s = a + b
    if s == 0:
        neg = (ca & 0x8000) and (cb & 0x8000)
        return 0x8000 if neg else 0x0000
    return H.brute_rn16(s)


def _finite_codes(rng, n):
    c = rng.integers(0, 65536, size=n).astype(np.uint16)
    return c[((c >> 9) & 63) != 63]


def test_add16_random_pairs_against_brute_force():
    rng = np.random.default_rng(200)
    a = _finite_codes(rng, 20000)
    b = _finite_codes(rng, 20000)
    n = min(len(a), len(b))
    a, b = a[:n], b[:n]
    got = oracle.add16(a, b)
    for x, y, g in zip(a.tolist(), b.tolist(), got.tolist()):
        assert _brute_add(x, y) == g, (hex(x), hex(y), hex(g))


def test_add16_exhaustive_window_against_brute_force():
    """All pairs whose exponent fields lie in a 4-wide window around 1.0, with
    every 37th mantissa: the region where rounding, ties and carries into the
    exponent all happen."""
    codes = []
    for e in range(29, 33):
        for m in range(0, 512, 37):
            codes.append((e << 9) | m)
    codes += [c | 0x8000 for c in codes]
    codes = np.array(codes, dtype=np.uint16)
    a = np.repeat(codes, len(codes))
    b = np.tile(codes, len(codes))
    got = oracle.add16(a, b)
    for x, y, g in zip(a.tolist(), b.tolist(), got.tolist()):
        assert _brute_add(x, y) == g, (hex(x), hex(y), hex(g))


def test_add16_subnormal_and_overflow_regions():
    rng = np.random.default_rng(201)
    small = np.concatenate([np.arange(0, 1024, dtype=np.uint16),
                            np.arange(0x8000, 0x8400, dtype=np.uint16)])
    a = rng.choice(small, 5000)
    b = rng.choice(small, 5000)
    got = oracle.add16(a, b)
    for x, y, g in zip(a.tolist(), b.tolist(), got.tolist()):
        assert _brute_add(x, y) == g
    big = np.arange(0x7C00, 0x7E00, dtype=np.uint16)
    a = rng.choice(big, 3000)
    b = rng.choice(big, 3000)
    got = oracle.add16(a, b)
    for x, y, g in zip(a.tolist(), b.tolist(), got.tolist()):
        assert _brute_add(x, y) == g


def test_swamping_threshold():
    """Sec. 2.3: with FP16 accumulation the smaller addend is truncated away
    once the magnitudes differ by more than 2^(mantissa+1) = 2^10."""
    for e in range(-20, 25):
        x = oracle.rn16(2.0 ** e)[()]
        for ratio_exp, lost in ((9, False), (10, True), (11, True), (12, True)):
            for frac in (1.0, 1.25, 1.5, 1.75):
                y_val = 2.0 ** (e - ratio_exp) * frac
                if ratio_exp == 10 and frac > 1.0:
                    continue        # ratio below 2^10: not covered by the claim
                y = oracle.rn16(y_val)[()]
                s = oracle.add16(x, y)[()]
                assert (s == x) == lost, (e, ratio_exp, frac)


def test_add16_invariants():
    rng = np.random.default_rng(202)
    a = _finite_codes(rng, 50000)
    b = _finite_codes(rng, 50000)
    n = min(len(a), len(b))
    a, b = a[:n], b[:n]
    ab, ba = oracle.add16(a, b), oracle.add16(b, a)
    assert np.array_equal(ab, ba)                                  # commutative
    neg = oracle.add16(a ^ 0x8000, b ^ 0x8000)
    nz = (ab & 0x7FFF) != 0
    assert np.array_equal(neg[nz], ab[nz] ^ 0x8000)                # odd
    zero = np.zeros_like(a)
    a_nz = a[(a & 0x7FFF) != 0]
    assert np.array_equal(oracle.add16(a_nz, zero[:len(a_nz)]), a_nz)   # x + 0 = x
    assert np.all(oracle.add16(a_nz, a_nz ^ 0x8000) == 0)         # x - x = +0
    # monotone in each argument
    va = oracle.p16_value(a)
    order = np.argsort(va, kind="stable")
    y = np.full(len(a), b[0], dtype=np.uint16)
    s = oracle.p16_value(oracle.add16(a[order], y))
    assert np.all(s[1:] >= s[:-1])
