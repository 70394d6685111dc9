"""Test-side helpers that are independent of the oracle's code.

The brute-force tables here enumerate every code of a format and decode it
from the bit-field definition with Python's exact rationals; rounding is then
a nearest-neighbour search over the sorted table.  That is a different
algorithm from the oracle's (integer significand shifting), so agreement pins
the oracle.
"""
import bisect
import os
from fractions import Fraction

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

P16_MAX = (2 - Fraction(1, 512)) * 2 ** 31
P8_MAX = Fraction(57344)


def parse_value(s):
    """Golden-file value syntax -> Fraction, or float for inf/nan/-0."""
    s = s.strip()
    if s in ("inf", "-inf", "nan", "-0.0"):
        return float(s)
    if s in ("max", "-max"):
        return -P16_MAX if s.startswith("-") else P16_MAX
    if "*2^" in s:
        a, b = s.split("*2^")
        return Fraction(a) * Fraction(2) ** int(b)
    return Fraction(s)


def read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append(line.split())
    return rows


def p8_fraction(c):
    """FP8 (1,5,2), bias 15: decode from the bit fields; None for Inf/NaN."""
    e, m = (c >> 2) & 31, c & 3
    if e == 31:
        return None
    v = Fraction(m, 4) * Fraction(2) ** -14 if e == 0 else (1 + Fraction(m, 4)) * Fraction(2) ** (e - 15)
    return -v if c & 0x80 else v


def p16_fraction(c):
    """FP16 (1,6,9), bias 31: decode from the bit fields; None for Inf/NaN."""
    e, m = (c >> 9) & 63, c & 511
    if e == 63:
        return None
    v = Fraction(m, 512) * Fraction(2) ** -30 if e == 0 else (1 + Fraction(m, 512)) * Fraction(2) ** (e - 31)
    return -v if c & 0x8000 else v


class Table:
    """Sorted non-negative finite values of a format with their codes."""

    def __init__(self, decode, ncodes, sign_bit):
        vals = {}
        for c in range(ncodes):
            if c & sign_bit:
                continue
            v = decode(c)
            if v is not None:
                vals[v] = c
        self.values = sorted(vals)
        self.codes = [vals[v] for v in self.values]
        self.sign_bit = sign_bit

    def neighbours(self, a):
        """Largest table value <= a and smallest >= a (a >= 0, in range)."""
        i = bisect.bisect_right(self.values, a) - 1
        lo = self.values[i]
        if lo == a:
            return i, i
        return i, i + 1

    def nearest_even(self, a):
        """Index of the nearest value to a >= 0, ties to the even code, or
        len(values) if a rounds beyond the largest value (overflow)."""
        top = self.values[-1]
        if a > top:
            # the next value above the top would be top + ulp(top); midpoint rule
            ulp = top - self.values[-2]
            mid = top + ulp / 2
            if a < mid:
                return len(self.values) - 1
            if a == mid:
                # tie: the top code is odd in these formats, the next is even
                return len(self.values)
            return len(self.values)
        i, j = self.neighbours(a)
        if i == j:
            return i
        lo, hi = self.values[i], self.values[j]
        if a - lo < hi - a:
            return i
        if a - lo > hi - a:
            return j
        return i if self.codes[i] % 2 == 0 else j


_P8 = None
_P16 = None


def p8_table():
    global _P8
    if _P8 is None:
        _P8 = Table(p8_fraction, 256, 0x80)
    return _P8


def p16_table():
    global _P16
    if _P16 is None:
        _P16 = Table(p16_fraction, 65536, 0x8000)
    return _P16


def brute_q8(x):
    """Round a float (FP32 value) to FP8 by nearest-neighbour search;
    finite overflow saturates."""
    if x != x:
        return 0x7F
    s = 0x80 if np.signbit(x) else 0
    if np.isinf(x):
        return s | 0x7C
    t = p8_table()
    i = t.nearest_even(abs(Fraction(float(x))))
    if i >= len(t.values):
        i = len(t.values) - 1
    return s | t.codes[i]


def brute_rn16(v):
    """Round an exact value (Fraction) to FP16 by nearest-neighbour search;
    overflow -> Inf.  Zero keeps no sign (callers handle -0)."""
    t = p16_table()
    s = 0x8000 if v < 0 else 0
    i = t.nearest_even(abs(v))
    if i >= len(t.values):
        return s | 0x7E00
    return s | t.codes[i]


def to_fraction16(code):
    return p16_fraction(int(code))


def p16_values(codes):
    """Vectorised decode of FP16 (1,6,9) codes from the bit fields (float64;
    Inf and NaN for exponent field 63)."""
    c = np.asarray(codes, dtype=np.uint16).astype(np.int64)
    e, m = (c >> 9) & 63, c & 511
    mag = np.where(e == 0, m * 2.0 ** -39, (512 + m) * np.exp2(np.maximum(e, 1) - 40.0))
    mag = np.where(e == 63, np.where(m == 0, np.inf, np.nan), mag)
    return np.where(c & 0x8000, -mag, mag)


def within_fast_bounds(C, lo, hi):
    """Per output: is the FP16 code C between the codes lo and hi in value
    (the fast mode's admissible results)?  NaN bounds admit only NaN."""
    v, a, b = p16_values(C), p16_values(lo), p16_values(hi)
    nan_b = np.isnan(a) | np.isnan(b)
    with np.errstate(invalid="ignore"):
        inside = (a <= v) & (v <= b)
    return np.where(nan_b, np.isnan(v), inside)
