"""Rounding identities the GPU kernels rely on, checked on the host in IEEE
single precision (numpy float32 arithmetic rounds to nearest even, as the
VALU does).  These pin the device algorithms, not the oracle."""
import numpy as np


def rne_significand10(u):
    """Integer round-to-nearest-even of float32 bit patterns to 10 significant
    bits: add half an ulp minus one plus the kept LSB, clear 14 bits."""
    return (u + np.uint32(0x1FFF) + ((u >> 14) & np.uint32(1))) & np.uint32(0xFFFFC000)


def veltkamp10(x):
    """c = x (2^14 + 1); hi = c - (c - x), each step rounded to float32."""
    c = (x * np.float32(16385.0)).astype(np.float32)
    d = (c - x).astype(np.float32)
    return (c - d).astype(np.float32)


def test_veltkamp_split_is_round_to_nearest_even_on_whole_binades():
    """Exhaustive over every significand of binades spanning the exact GEMM's
    guarded domain (unscaled FP16 values: normal from 2^-30 up to the 2^31
    bound of the guard), both signs; ties (frequent for sums of FP8 products)
    must go to even."""
    m = np.arange(1 << 23, dtype=np.uint32)
    for e in (127 - 30, 127 - 1, 127, 127 + 30):
        for sign in (0, 1):
            u = (np.uint32(sign) << np.uint32(31)) | (np.uint32(e) << np.uint32(23)) | m
            x = u.view(np.float32)
            assert np.array_equal(veltkamp10(x).view(np.uint32), rne_significand10(u)), e


def test_veltkamp_split_keeps_short_values():
    """Values with at most 10 significant bits (e.g. FP16 subnormal sums,
    k * 2^-39 with k < 512) pass through unchanged."""
    k = np.arange(1, 1 << 10, dtype=np.float64)
    for scale in (2.0 ** -39, 2.0 ** -20, 2.0 ** 10):
        x = (k * scale).astype(np.float32)
        assert np.array_equal(veltkamp10(x), x)
        assert np.array_equal(veltkamp10(-x), -x)
    assert veltkamp10(np.float32([0.0]))[0] == 0.0


# --- products of two FP16 values (the FP16-operand GEMM) -------------------

def fp16_operands(exp, neg=False):
    """Every FP16 normal value 2^exp (1 + m/512), m = 0..511, as float32."""
    v = (512.0 + np.arange(512)) * 2.0 ** (exp - 9)
    return (-v if neg else v).astype(np.float32)


def rn16_reference(p):
    """Exact products (float64) rounded to the FP16 grid by integer
    arithmetic: quantum 2^(max(E, -30) - 9) for |p| in [2^E, 2^(E+1)), ties
    to even; Inf from the largest FP16 value's midpoint on."""
    p = np.asarray(p, np.float64)
    e = np.floor(np.log2(np.where(p == 0, 1.0, np.abs(p))))
    q = np.exp2(np.maximum(e, -30.0) - 9.0)
    r = np.rint(p / q) * q
    r = np.where(np.abs(r) >= 2.0 ** 32, np.inf * np.sign(p), r)
    return np.where(p == 0, 0.0, r)


def fma32(a, b, c):
    """fmaf(a, b, c) for float32 a, b, c when a b is exact in float64 and
    a b + c needs at most 53 bits: one rounding of the float64 result."""
    return (a.astype(np.float64) * b.astype(np.float64) + c.astype(np.float64)).astype(np.float32)


def test_fp16_product_veltkamp_split_is_rn16():
    """c = a (b (2^14 + 1)), hi = c + fma(a, b, -c) rounds the exact product
    of two FP16 values to FP16 (nearest even) whenever it is at least 2^-30
    (and below the guard's 2^31): every pair of significands, both sign
    combinations, products from 2^-30 to 2^31."""
    for ea, eb in ((-15, -15), (-30, 0), (0, 0), (-1, -1), (15, 14), (7, -20)):
        for na in (False, True):
            a = fp16_operands(ea, na)[:, None]
            b = fp16_operands(eb)[None, :]
            bs = (b * np.float32(16385.0)).astype(np.float32)
            assert np.array_equal(bs.astype(np.float64), b.astype(np.float64) * 16385.0)
            c = (a * bs).astype(np.float32)
            hi = (c + fma32(a, b, -c)).astype(np.float32)
            exact = a.astype(np.float64) * b.astype(np.float64)
            assert np.array_equal(hi.astype(np.float64), rn16_reference(exact)), (ea, eb, na)
    # a zero product gives +0 whatever the signs
    for a, b in ((0.0, 3.0), (-0.0, 3.0), (0.0, -3.0), (-2.0, 0.0)):
        a32, b32 = np.float32([a]), np.float32([b])
        c = (a32 * (b32 * np.float32(16385.0))).astype(np.float32)
        hi = (c + fma32(a32, b32, -c)).astype(np.float32)
        assert hi.view(np.uint32)[0] == 0


def rn16_product_plain(p):
    """The plain-value magic-number rounding of an exact float32 product."""
    e = p.view(np.uint32) & np.uint32(0x7F800000)
    e = np.maximum(e, np.uint32(97 << 23))
    magic = (e + np.uint32(14 << 23) + np.uint32(0x00400000)).view(np.float32)
    return ((p + magic).astype(np.float32) - magic).astype(np.float32)


def rn16_product_scaled(p64):
    """The 2^64-domain variant: clamp the exponent to [34, 113], round with
    the magic number, return the result times 2^32 (the 2^96 domain)."""
    e = p64.view(np.uint32) & np.uint32(0x7F800000)
    e = np.minimum(np.maximum(e, np.uint32(161 << 23)), np.uint32(240 << 23))
    magic = (e + np.uint32(14 << 23) + np.uint32(0x00400000)).view(np.float32)
    with np.errstate(over="ignore", invalid="ignore"):
        r = ((p64 + magic).astype(np.float32) - magic).astype(np.float32)
        return (r * np.float32(2.0 ** 32)).astype(np.float32)


def fp16_subnormals():
    return (np.arange(1, 512) * 2.0 ** -39).astype(np.float32)


def test_fp16_product_magic_rounding_plain():
    """The guarded path's product rounding: every significand pair over
    exponents that put products in FP16's subnormal range (fixed step 2^-39),
    across the 2^-30 boundary and in the normal range; FP16 subnormal
    operands too."""
    cases = [(-30, -30), (-20, -12), (-16, -15), (-15, -15), (0, 0), (15, 14)]
    for ea, eb in cases:
        for na in (False, True):
            a = fp16_operands(ea, na)[:, None]
            b = fp16_operands(eb)[None, :]
            got = rn16_product_plain((a * b).astype(np.float32))
            exact = a.astype(np.float64) * b.astype(np.float64)
            assert np.array_equal(got.astype(np.float64), rn16_reference(exact)), (ea, eb)
    a = fp16_subnormals()[:, None]
    for eb in (-10, 0, 20):
        b = fp16_operands(eb)[None, :]
        got = rn16_product_plain((a * b).astype(np.float32))
        assert np.array_equal(got.astype(np.float64),
                              rn16_reference(a.astype(np.float64) * b.astype(np.float64))), eb


def test_fp16_product_magic_rounding_scaled():
    """The 2^96-domain product rounding of the safe path (operands scaled by
    2^48 and 2^16): subnormal-range, normal and overflowing products (those
    at or beyond the largest FP16 value's midpoint become Inf), up to the
    largest FP16 operands, and FP16 subnormal operands."""
    cases = [(-30, -30), (-16, -15), (0, 0), (15, 15), (16, 16), (31, 31), (31, -39 + 9)]
    for ea, eb in cases:
        for na in (False, True):
            a = fp16_operands(ea, na)[:, None]
            b = fp16_operands(eb)[None, :]
            p64 = ((a * np.float32(2.0 ** 48)) * (b * np.float32(2.0 ** 16))).astype(np.float32)
            got = rn16_product_scaled(p64).astype(np.float64) * 2.0 ** -96
            exact = a.astype(np.float64) * b.astype(np.float64)
            assert np.array_equal(got, rn16_reference(exact)), (ea, eb, na)
    a = fp16_subnormals()[:, None]
    b = fp16_operands(-5)[None, :]
    p64 = ((a * np.float32(2.0 ** 48)) * (b * np.float32(2.0 ** 16))).astype(np.float32)
    got = rn16_product_scaled(p64).astype(np.float64) * 2.0 ** -96
    assert np.array_equal(got, rn16_reference(a.astype(np.float64) * b.astype(np.float64)))
    # zero, Inf and NaN pass through
    z = rn16_product_scaled(np.float32([0.0, np.inf, -np.inf, np.nan]))
    assert z[0] == 0.0 and z[1] == np.inf and z[2] == -np.inf and np.isnan(z[3])


def test_guarded_fp16_encode_round_trips_every_code():
    """The guarded paths' encoder (x 2^-96 in float32 -- an FP32 subnormal
    for FP16 subnormals --, its bits 14-28 as exponent and significand, bit
    31 as sign): every finite FP16 code below 2^32, both signs, decoded by
    the oracle's definition and encoded with float32 arithmetic that keeps
    subnormals, gives the code back (-0 included), with zero upper bits."""
    import oracle
    codes = np.arange(1 << 16, dtype=np.uint32)
    finite = (codes & 0x7E00) != 0x7E00
    codes = codes[finite]
    x = oracle.p16_value(codes.astype(np.uint16)).astype(np.float32)
    assert np.all(np.abs(x) < np.float32(2.0 ** 32))
    y = x * np.float32(2.0 ** -96)
    # the scaling is exact (the FP32 subnormal range included)
    assert np.array_equal(y.astype(np.float64) * 2.0 ** 96, x.astype(np.float64))
    b = y.view(np.uint32)
    enc = ((b >> np.uint32(14)) & np.uint32(0x7FFF)) | ((b >> np.uint32(16)) & np.uint32(0xFFFF8000))
    assert np.array_equal(enc, codes)
