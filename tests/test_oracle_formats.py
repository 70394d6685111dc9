"""Pins for the oracle's number formats (Sec. 2.2): FP8 (1,5,2) and FP16 (1,6,9).

What pins the oracle here (none of it re-uses the oracle's own code):
* torch's float8_e5m2 decode and cast (an independent library
  implementation of a 1-5-2 format with bias 15 and subnormals) agrees with
  every finite FP8 code and with round-to-nearest-even in the finite range;
* brute-force nearest-neighbour search over all codes decoded with exact
  rationals from the bit fields;
* hand-worked cases in tests/golden/rounding_cases.txt.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from tests import helpers as H


def test_p8_decode_matches_torch_e5m2():
    codes = np.arange(256, dtype=np.uint8)
    ours = oracle.p8_value(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e5m2).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])
    assert np.array_equal(np.signbit(ours[~nan]), np.signbit(ref[~nan]))


def test_p8_value_set():
    vals = oracle.p8_value(np.arange(256, dtype=np.uint8))
    finite = vals[np.isfinite(vals)]
    assert len(finite) == 248                      # 256 - Inf/NaN field
    assert len(set(finite.tolist())) == 247        # +0 and -0 are one value
    assert finite.max() == 57344.0
    assert finite[finite > 0].min() == 2.0 ** -16
    # every code decodes to its bit-field value
    for c in range(256):
        f = H.p8_fraction(c)
        if f is not None:
            assert Fraction(float(vals[c])) == f
    # positive codes are ordered by value
    pos = vals[:0x7C]
    assert np.all(np.diff(pos) > 0)


def test_p16_value_set_and_roundtrip():
    codes = np.arange(65536, dtype=np.uint32)
    vals = np.array([oracle.lib().orc_p16_value(int(c)) for c in codes])
    fin = np.isfinite(vals)
    assert fin.sum() == 65536 - 2 * 512            # field 63 holds Inf/NaN
    assert vals[fin].max() == 4290772992.0         # (2 - 2^-9) * 2^31
    assert vals[(vals > 0)].min() == 2.0 ** -39
    assert np.all(np.diff(vals[:0x7E00]) > 0)      # ordered
    for c in range(0, 65536, 97):                  # bit-field definition
        f = H.p16_fraction(c)
        if f is not None:
            assert Fraction(float(vals[c])) == f
    back = oracle.rn16(vals[fin])
    assert np.array_equal(back, codes[fin].astype(np.uint16))


@pytest.mark.parametrize("row", H.read_golden("rounding_cases.txt"))
def test_golden_rounding(row):
    op = row[0]
    if op == "q8":
        x = float(H.parse_value(row[1])) if not isinstance(H.parse_value(row[1]), float) else H.parse_value(row[1])
        x32 = np.float32(x)
        assert int(oracle.q8(float(x32))) == int(row[2], 16)
        assert H.brute_q8(float(x32)) == int(row[2], 16) or math.isnan(x)
    elif op == "add16":
        a, b = H.parse_value(row[1]), H.parse_value(row[2])
        ca = oracle.rn16(float(a))[()]
        cb = oracle.rn16(float(b))[()]
        assert int(oracle.add16(ca, cb)) == int(row[3], 16)
    else:
        raise AssertionError(op)


def test_q8_matches_torch_cast_in_finite_range():
    rng = np.random.default_rng(100)
    # cover every binade from far below the subnormals to the top of the range
    e = rng.uniform(-30.0, 16.0, size=200_000)
    x = (np.sign(rng.standard_normal(e.size)) * np.exp2(e)).astype(np.float32)
    x = x[np.abs(x) < 61440.0]       # torch overflows to Inf from here on
    # add exact ties: midpoints between neighbouring finite values
    vals = np.unique(oracle.p8_value(np.arange(0x7C, dtype=np.uint8)))
    mids = ((vals[1:] + vals[:-1]) / 2).astype(np.float32)
    x = np.concatenate([x, mids, -mids])
    ref = torch.from_numpy(x).to(torch.float8_e5m2).view(torch.uint8).numpy()
    ours = oracle.fp8_quantize(x)
    assert np.array_equal(ours, ref)


def test_q8_brute_force_nearest_including_saturation():
    rng = np.random.default_rng(101)
    e = rng.uniform(-20.0, 20.0, size=3000)
    x = (np.sign(rng.standard_normal(e.size)) * np.exp2(e)).astype(np.float32)
    ours = oracle.fp8_quantize(x)
    for xi, qi in zip(x.tolist(), ours.tolist()):
        assert H.brute_q8(xi) == qi, xi


def test_q8_scale_multiplies_in_fp32():
    rng = np.random.default_rng(102)
    x = rng.standard_normal(5000).astype(np.float32) * np.float32(1e-3)
    s = np.float32(1000.0)
    ours = oracle.fp8_quantize(x, scale=float(s))
    ref = torch.from_numpy(x * s).to(torch.float8_e5m2).view(torch.uint8).numpy()
    assert np.array_equal(ours, ref)


def test_q8_from_fp16_codes_is_single_rounding():
    codes = np.arange(65536, dtype=np.uint16)
    vals = np.array([oracle.lib().orc_p16_value(int(c)) for c in codes])
    ok = np.isfinite(vals) & (np.abs(vals) < 61440.0)
    ours = oracle.fp8_quantize(codes)
    # every FP16 value is an FP32 value, so a single FP32 -> FP8 cast is the
    # same single rounding
    ref = torch.from_numpy(vals.astype(np.float32)).to(torch.float8_e5m2).view(torch.uint8).numpy()
    assert np.array_equal(ours[ok], ref[ok])
    big = np.isfinite(vals) & (np.abs(vals) >= 61440.0)
    assert np.all((ours[big] & 0x7F) == 0x7B)


def test_all_fp8_products_are_exact_in_fp16():
    """Sec. 2.3 multiplies in FP8 and accumulates in FP16; every product of two
    FP8 values fits FP16 exactly (3-bit x 3-bit significands, exponents within
    range), so the product step never rounds."""
    a = np.repeat(np.arange(256, dtype=np.uint8), 256)
    b = np.tile(np.arange(256, dtype=np.uint8), 256)
    va, vb = oracle.p8_value(a), oracle.p8_value(b)
    with np.errstate(invalid="ignore"):  # Inf x 0 -> NaN among the special codes
        prod = va * vb                  # exact in float64
    codes = oracle.mul8(a, b)
    got = oracle.p16_value(codes)
    fin = np.isfinite(prod)
    assert np.array_equal(got[fin], prod[fin])
    assert np.array_equal(np.isnan(got), np.isnan(prod))
    assert np.array_equal(got[np.isinf(prod)], prod[np.isinf(prod)])


def test_fp16_quantize_brute_force_nearest():
    """FP32 -> FP16 round-to-nearest-even, checked by nearest-neighbour search
    over all FP16 codes, across the subnormal range, ties and overflow."""
    rng = np.random.default_rng(103)
    e = rng.uniform(-45.0, 34.0, size=4000)
    x = (np.sign(rng.standard_normal(e.size)) * np.exp2(e)).astype(np.float32)
    vals = np.unique(oracle.p16_value(np.arange(0x7E00, dtype=np.uint16)))
    mids = ((vals[1:] + vals[:-1]) / 2).astype(np.float32)      # exact ties
    x = np.concatenate([x, rng.choice(mids, 2000), np.float32([0.0, -0.0, np.inf, -np.inf])])
    got = oracle.fp16_quantize(x)
    for xi, gi in zip(x.tolist(), got.tolist()):
        if xi == 0:
            ref = 0x8000 if np.signbit(xi) else 0
        elif np.isinf(xi):
            ref = 0xFE00 if xi < 0 else 0x7E00
        else:
            ref = H.brute_rn16(Fraction(xi))
        assert ref == gi, (xi, hex(gi), hex(ref))
