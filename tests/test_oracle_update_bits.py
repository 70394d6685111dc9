"""Bit-level pin of the oracle's FP16 SGD update (Sec. 2.2 Fig. 2(b): the
L2-Reg, Momentum-Acc and Weight-Upd AXPYs; Sec. 2.3 Eq. (1); Sec. 4.3).

The update is recomputed here from its definition with nothing shared with
`oracle/ops.c` except the Philox block function (pinned separately against
rocRAND's header) and the FP8 quantizer (pinned against brute-force search):

* FP16 codes are decoded from the bit fields with exact rationals;
* each AXPY is the exact rational a*b + c rounded once to float32 (a fused
  multiply-add), with IEEE's zero-sign rule for exact zeros;
* stochastic rounding is Eq. (1) on the rational value: the magnitude is
  rounded up by one FP16 step 2^(e-9) (2^-39 below 2^-30) iff the 16-bit
  uniform is below floor(fraction * 2^16);
* the random bits are the eight 16-bit halves (low half first) of the
  Philox4x32-10 block with counter (pair lo, pair hi, offset lo, offset hi) and
  key (seed lo, seed hi); element i takes halves 3 (i mod 2) + 0, 1, 2.

Mutated versions of this formulation (the slips a shared misreading could
hide: another uniform layout, high half first, swapped counter words or key
halves, an unfused AXPY, L2-Reg after Momentum-Acc) must each disagree with
the oracle, so the match is not an accident of the data.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
from tests.helpers import brute_rn16, p16_fraction

TWO = Fraction(2)
P16_MAX = (2 - Fraction(1, 512)) * TWO ** 31


# ---- float32 and FP16 as exact rationals ------------------------------------

def f32_fraction(x):
    return Fraction(float(np.float32(x)))


def rn32(fr):
    """Round a rational to the nearest float32, ties to even.  The update's
    operands keep every result inside float32's normal range or at zero."""
    if fr == 0:
        return np.float32(0.0)
    s = -1 if fr < 0 else 1
    a = abs(fr)
    e = math.floor(math.log2(a))
    while TWO ** e > a:
        e -= 1
    while TWO ** (e + 1) <= a:
        e += 1
    assert -126 <= e <= 127, "outside the normal float32 range"
    t = a / TWO ** (e - 23)
    n = math.floor(t)
    r = t - n
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return np.float32(s * float(n * TWO ** (e - 23)))


def fma32(a, b, c, fused=True):
    """float32 fused multiply-add a*b + c (one rounding); fused=False rounds
    the product first (the mutation of an unfused AXPY)."""
    a, b, c = np.float32(a), np.float32(b), np.float32(c)
    if not (np.isfinite(a) and np.isfinite(b) and np.isfinite(c)):
        with np.errstate(invalid="ignore", over="ignore"):
            return np.float32(float(a) * float(b) + float(c))
    prod = f32_fraction(a) * f32_fraction(b)
    if not fused:
        p32 = rn32(prod) if prod != 0 else np.float32(0.0)
        if prod == 0:
            p32 = np.float32(-0.0) if (np.signbit(a) != np.signbit(b)) else np.float32(0.0)
        return fma32(np.float32(1.0), p32, c)
    total = prod + f32_fraction(c)
    if total == 0:
        # IEEE: an exact zero sum is +0 unless both addends are zeros of
        # negative sign (the product's sign is the xor of the factors' signs)
        prod_neg_zero = prod == 0 and (np.signbit(a) != np.signbit(b))
        if prod_neg_zero and f32_fraction(c) == 0 and np.signbit(c):
            return np.float32(-0.0)
        return np.float32(0.0)
    return rn32(total)


def decode16(code):
    """FP16 (1,6,9) code -> float32 value (every finite FP16 value is one)."""
    code = int(code)
    v = p16_fraction(code)
    if v is None:
        if code & 0x1FF:
            return np.float32(np.nan)
        return np.float32(-np.inf if code & 0x8000 else np.inf)
    if v == 0:
        return np.float32(-0.0 if code & 0x8000 else 0.0)
    return np.float32(float(v))


def sr16(x, u):
    """Eq. (1) with k' = 23 (x is a float32) and k = 9, step 2^-39 below 2^-30;
    results beyond the largest finite FP16 value are Inf; NaN -> 0x7F00."""
    x = np.float32(x)
    sign = 0x8000 if np.signbit(x) else 0
    if np.isnan(x):
        return 0x7F00
    if np.isinf(x):
        return sign | 0x7E00
    a = f32_fraction(abs(x))
    if a == 0:
        return sign
    e = math.floor(math.log2(a))
    while TWO ** e > a:
        e -= 1
    while TWO ** (e + 1) <= a:
        e += 1
    q = TWO ** -39 if a < TWO ** -30 else TWO ** (e - 9)
    t = a / q
    n = math.floor(t)
    F = math.floor((t - n) * 65536)
    r = (n + (1 if u < F else 0)) * q
    if r > P16_MAX:
        return sign | 0x7E00
    code = brute_rn16(r)          # r is an FP16 value: the search finds it exactly
    assert p16_fraction(code) == r
    return sign | code


# ---- the random bits ----------------------------------------------------------

def halves(pair, seed, offset, *, high_first=False, swap_ctr=False, swap_key=False):
    ctr = [pair & 0xFFFFFFFF, pair >> 32, offset & 0xFFFFFFFF, offset >> 32]
    if swap_ctr:
        ctr = ctr[2:] + ctr[:2]
    key = [seed & 0xFFFFFFFF, seed >> 32]
    if swap_key:
        key = key[::-1]
    words = oracle.philox4x32_10(ctr, key)
    h = []
    for w in words:
        lo, hi = int(w) & 0xFFFF, int(w) >> 16
        h += [hi, lo] if high_first else [lo, hi]
    return h


# ---- the update, written from its definition ----------------------------------

def update_element(i, w, g, v, lr, mu, wd, seed, offset, mut=None):
    """Returns (w', v' or None) codes of element i."""
    mut = mut or ""
    h = halves(i >> 1, seed, offset, high_first=mut == "high_first",
               swap_ctr=mut == "swap_ctr", swap_key=mut == "swap_key")
    base = 4 * (i & 1) if mut == "layout4" else 3 * (i & 1)
    u = h[base: base + 3]
    fused = mut != "unfused"
    wf, gf = decode16(w), decode16(g)
    lr, mu, wd = np.float32(lr), np.float32(mu), np.float32(wd)
    if v is None:
        g1 = sr16(fma32(wd, wf, gf, fused), u[0])
        w1 = sr16(fma32(-lr, decode16(g1), wf, fused), u[2])
        return w1, None
    vf = decode16(v)
    if mut == "wd_after_momentum":
        v1 = sr16(fma32(mu, vf, gf, fused), u[1])
        s1 = sr16(fma32(wd, wf, decode16(v1), fused), u[0])
        w1 = sr16(fma32(-lr, decode16(s1), wf, fused), u[2])
        return w1, v1
    g1 = sr16(fma32(wd, wf, gf, fused), u[0])
    v1 = sr16(fma32(mu, vf, decode16(g1), fused), u[1])
    w1 = sr16(fma32(-lr, decode16(v1), wf, fused), u[2])
    return w1, v1


def independent_update(w, g, v, lr, mu, wd, seed, offset, mut=None):
    n = w.size
    ow = np.empty(n, np.uint16)
    ov = None if v is None else np.empty(n, np.uint16)
    for i in range(n):
        a, b = update_element(i, w[i], g[i], None if v is None else v[i], lr, mu, wd,
                              seed, offset, mut)
        ow[i] = a
        if ov is not None:
            ov[i] = b
    return ow, ov


# ---- inputs ---------------------------------------------------------------------

def _codes(x):
    return oracle.fp16_quantize(np.asarray(x, np.float32))


def special_inputs(rng, n):
    """Typical values plus zeros of both signs, FP16 subnormals, values at the
    top of the range (the update overflows to Inf), Inf and NaN."""
    w = _codes(rng.standard_normal(n) * 0.05)
    g = _codes(rng.standard_normal(n) * 1e-3)
    v = _codes(rng.standard_normal(n) * 1e-3)
    spec = np.array([0x0000, 0x8000, 0x0001, 0x8001, 0x01FF, 0x0200, 0x81FF,
                     0x7DFF, 0xFDFF, 0x7E00, 0xFE00, 0x7F00, 0x3E00, 0xBE00], np.uint16)
    for arr in (w, g, v):
        k = rng.integers(0, n, 40)
        arr[k] = spec[rng.integers(0, spec.size, 40)]
    # tiny steps: lr * v below 2^-30 lands the sum in the subnormal range
    k = rng.integers(0, n, 20)
    w[k] = rng.integers(0, 0x0200, 20).astype(np.uint16)
    # all three operands in the subnormal range: subnormal results
    k = rng.integers(0, n, 20)
    for arr in (w, g, v):
        arr[k] = rng.integers(0, 0x0200, 20).astype(np.uint16) | \
            (rng.integers(0, 2, 20) << 15).astype(np.uint16)
    return w, g, v


CASES = [
    # n (odd), lr, momentum, weight decay, seed, offset, with v, with w8
    dict(n=301, lr=0.1, mu=0.9, wd=1e-4, seed=7, offset=0, v=True, w8=True),
    dict(n=257, lr=0.1, mu=0.0, wd=0.0, seed=1, offset=3, v=False, w8=True),
    dict(n=199, lr=0.03125, mu=0.9, wd=5e-4, seed=(1 << 40) + 12345,
         offset=(1 << 33) + 17, v=True, w8=False),
    dict(n=151, lr=2.5, mu=0.5, wd=0.25, seed=2 ** 64 - 1, offset=2 ** 63 + 5, v=True,
         w8=True),
    dict(n=129, lr=1e-3, mu=0.0, wd=1e-2, seed=99, offset=(1 << 32), v=False, w8=False),
]


def _oracle(case, w, g, v):
    return oracle.sr_weight_update(w, g, v if case["v"] else None, lr=case["lr"],
                                   momentum=case["mu"], weight_decay=case["wd"],
                                   seed=case["seed"], offset=case["offset"],
                                   want_w8=case["w8"])


@pytest.mark.parametrize("ci", range(len(CASES)))
def test_update_bit_for_bit(ci):
    case = CASES[ci]
    rng = np.random.default_rng(960 + ci)
    w, g, v = special_inputs(rng, case["n"])
    ow, ov, o8 = _oracle(case, w, g, v)
    iw, iv = independent_update(w, g, v if case["v"] else None, case["lr"], case["mu"],
                                case["wd"], case["seed"], case["offset"])
    bad = np.flatnonzero(iw != ow)
    assert bad.size == 0, [(int(i), hex(w[i]), hex(g[i]), hex(iw[i]), hex(ow[i]))
                           for i in bad[:5]]
    if case["v"]:
        assert np.array_equal(iv, ov)
    else:
        assert ov is None
    if case["w8"]:
        assert np.array_equal(o8, oracle.fp8_quantize(ow))
    else:
        assert o8 is None
    # the special codes reached every branch: Inf, NaN, zero and subnormal outputs
    assert np.any((ow & 0x7FFF) == 0x7E00) and np.any(ow == 0x7F00)
    assert np.any(((ow & 0x7E00) == 0) & ((ow & 0x1FF) != 0))


def test_update_long_run_of_typical_elements():
    """Two thousand typical elements (the benchmark update's distributions),
    every one bit for bit."""
    rng = np.random.default_rng(970)
    n = 2001
    w = _codes(rng.standard_normal(n) * 0.02)
    g = _codes(rng.standard_normal(n) * 1e-4)
    v = _codes(rng.standard_normal(n) * 1e-4)
    ow, ov, _ = oracle.sr_weight_update(w, g, v, lr=0.1, momentum=0.9, weight_decay=1e-4,
                                        seed=7, offset=11, want_w8=False)
    iw, iv = independent_update(w, g, v, 0.1, 0.9, 1e-4, 7, 11)
    assert np.array_equal(iw, ow) and np.array_equal(iv, ov)


MUTATIONS = ["layout4", "high_first", "swap_ctr", "swap_key", "unfused",
             "wd_after_momentum"]


def _plant_unfused_witnesses(w, g, v, wd, seed, offset, idx, rng):
    """Rewrite elements idx so that the first AXPY, fma(wd, w, g), decides its
    stochastic rounding differently when the product is rounded to float32
    before the addition.  In FP16's normal range Eq. (1) rounds a float32 up
    iff its 14 discarded significand bits m satisfy 4 m > u (F = 4 m exactly),
    so a one-ulp float32 difference flips the result when u falls between the
    two.  The search is vectorised: the product of an FP32 scalar and an FP16
    value and its sum with an FP16 value within ten binades are exact in
    float64, so float64 -> float32 gives the fused result."""
    wd32 = np.float32(wd)
    for i in idx:
        u = halves(int(i) >> 1, seed, offset)[3 * (int(i) & 1)]
        for _ in range(50):
            wc = (rng.integers(25 << 9, 36 << 9, 1 << 16) |
                  (rng.integers(0, 2, 1 << 16) << 15)).astype(np.uint16)
            gc = (rng.integers(18 << 9, 29 << 9, 1 << 16) |
                  (rng.integers(0, 2, 1 << 16) << 15)).astype(np.uint16)
            wv = oracle.p16_value(wc)
            gv = oracle.p16_value(gc)
            prod = np.float64(wd32) * wv
            fused = (prod + gv).astype(np.float32)
            unfused = (prod.astype(np.float32) + gv.astype(np.float32)).astype(np.float32)

            def sr_bits(x):
                b = x.view(np.uint32)
                up = 4 * (b & np.uint32(0x3FFF)) > np.uint32(u)
                return (b & np.uint32(0xFFFFC000)) + up.astype(np.uint32) * np.uint32(0x4000)

            ok = (np.abs(fused) >= 2.0 ** -29) & (sr_bits(fused) != sr_bits(unfused))
            if ok.any():
                k = int(np.flatnonzero(ok)[0])
                w[i], g[i], v[i] = wc[k], gc[k], 0
                break
        else:
            raise AssertionError("no witness found")


@pytest.mark.parametrize("mut", MUTATIONS)
def test_mutations_are_detected(mut):
    """Each plausible slip changes some bits of the result, so the bit-for-bit
    agreement above pins these choices.  Random data detects all but the
    unfused AXPY (a one-ulp float32 difference decides a stochastic rounding
    with probability ~2^-14); for it, elements are planted where the uniform
    falls between the two outcomes."""
    rng = np.random.default_rng(980)
    n = 400
    w = _codes(rng.standard_normal(n) * 0.05)
    g = _codes(rng.standard_normal(n) * 1e-2)
    v = _codes(rng.standard_normal(n) * 1e-2)
    lr, mu, wd, seed, off = 0.1, 0.9, 0.01, (3 << 32) + 5, (1 << 32) + 2
    _plant_unfused_witnesses(w, g, v, wd, seed, off, [5, 6, 101, 398], rng)
    ow, ov, _ = oracle.sr_weight_update(w, g, v, lr=lr, momentum=mu, weight_decay=wd,
                                        seed=seed, offset=off, want_w8=False)
    iw, iv = independent_update(w, g, v, lr, mu, wd, seed, off)
    assert np.array_equal(iw, ow) and np.array_equal(iv, ov)
    mw, mv = independent_update(w, g, v, lr, mu, wd, seed, off, mut=mut)
    assert not (np.array_equal(mw, ow) and np.array_equal(mv, ov)), mut


def test_header_documents_this_update():
    """The public header states the AXPY order and random-bit layout that the
    formulation above recomputes."""
    import os
    import re
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                        "include", "fp8train.h")
    with open(path) as f:
        doc = re.sub(r"\s+", " ", re.sub(r"\n\s*\*\s?", " ", f.read()))
    seg = doc[doc.index("sr_weight_update -- "):doc.index("int sr_weight_update(")]
    for phrase in ("g' = SR(fmaf(weight_decay, w[i], g[i]))",
                   "v' = SR(fmaf(momentum, v[i], g'))",
                   "w' = SR(fmaf(-lr, v', w[i]))",
                   "key = (seed low, seed high) and counter = (i/2 low, i/2 high, offset low, "
                   "offset high)",
                   "eight 16-bit uniforms (low half first)",
                   "element i uses uniforms 3*(i%2)+0, +1, +2 for g', v', w'"):
        assert phrase in seg, phrase
