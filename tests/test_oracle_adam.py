"""Pins for the oracle's ADAM update in P16 with stochastic rounding (Sec. 3:
ADAM with FP8 GEMMs and FP16 weight updates; Kingma & Ba's algorithm with the
AXPYs of Sec. 2.2 rounded by Eq. (1)).

* the bias-corrected step size equals lr sqrt(1 - beta2^t) / (1 - beta1^t)
  computed exactly, to within one FP32 rounding;
* an independent formulation -- exact rational arithmetic for the fused
  multiply-adds and Eq. (1), numpy float32 for the other IEEE operations --
  reproduces the oracle bit for bit;
* on the first step the update is lr times the gradient's sign (m/sqrt(v) is
  +-1 for |g| >> eps), as Kingma & Ba note;
* stochastic rounding keeps updates far below one FP16 step in expectation
  (the reason Sec. 4.3 rounds the updates stochastically), where nearest
  rounding would drop them;
* over several steps the trajectory follows float64 ADAM.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle

U16 = 65536


def _f(x):
    return Fraction(float(x))


def rn32(fr):
    """Round a non-zero rational to the nearest float32, ties to even (normal
    range only)."""
    if fr == 0:
        return np.float32(0.0)
    s = -1 if fr < 0 else 1
    a = abs(fr)
    e = math.floor(math.log2(a))
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    assert -126 <= e <= 127
    t = a / Fraction(2) ** (e - 23)          # in [2^23, 2^24)
    n = math.floor(t)
    r = t - n
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return np.float32(s * float(n * Fraction(2) ** (e - 23)))


def fma32(a, b, c):
    return rn32(_f(a) * _f(b) + _f(c))


def sr16(x, u):
    """Eq. (1) on float32 x with 16-bit uniform u (finite, |x| < 2^32)."""
    a = abs(_f(x))
    if a == 0:
        return float(x)
    e = math.floor(math.log2(a))
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    q = Fraction(2) ** -39 if a < Fraction(2) ** -30 else Fraction(2) ** (e - 9)
    t = a / q
    n = math.floor(t)
    F = math.floor((t - n) * U16)
    r = float((n + (1 if u < F else 0)) * q)
    return math.copysign(r, float(x))


def uniforms(i, seed, offset):
    words = oracle.philox4x32_10([i // 2 & 0xFFFFFFFF, i // 2 >> 32, offset & 0xFFFFFFFF,
                                  offset >> 32], [seed & 0xFFFFFFFF, seed >> 32])
    u = []
    for w in words:
        u += [int(w) & 0xFFFF, int(w) >> 16]
    return u[4 * (i % 2): 4 * (i % 2) + 4]


def _p16(x):
    return oracle.fp16_quantize(np.asarray(x, np.float32))


@pytest.mark.parametrize("t", [1, 2, 10, 1000, 10 ** 6])
def test_step_size_closed_form(t):
    lr, b1, b2 = np.float32(1e-3), np.float32(0.9), np.float32(0.999)
    got = oracle.adam_step_size(lr, b1, b2, t)
    # exact value within float64 evaluation error, compared after rounding
    ex = float(lr) * math.sqrt(1 - float(b2) ** t) / (1 - float(b1) ** t)
    assert abs(got - ex) <= 2 * np.spacing(np.float32(ex))


def test_independent_formulation():
    rng = np.random.default_rng(950)
    n = 64
    w = _p16(rng.standard_normal(n) * 0.05)
    g = _p16(rng.standard_normal(n) * 1e-3)
    m = _p16(rng.standard_normal(n) * 1e-4)
    v = _p16(np.abs(rng.standard_normal(n)) * 1e-6)
    lr, b1, b2, eps, wd, t, seed, off = 1e-3, 0.9, 0.999, 1e-8, 1e-4, 7, 12345, 3
    ow, om, ov, o8 = oracle.adam_update(w, g, m, v, lr=lr, beta1=b1, beta2=b2, eps=eps,
                                        weight_decay=wd, t=t, seed=seed, offset=off)
    alpha = np.float32(oracle.adam_step_size(lr, b1, b2, t))
    b1, b2, eps, wd = (np.float32(x) for x in (b1, b2, eps, wd))
    c1, c2 = np.float32(1) - b1, np.float32(1) - b2
    val = oracle.p16_value
    for i in range(n):
        h = uniforms(i, seed, off)
        wf, gf, mf, vf = (np.float32(val(a[i])) for a in (w, g, m, v))
        g1 = np.float32(sr16(fma32(wd, wf, gf), h[0]))
        m1 = np.float32(sr16(fma32(b1, mf, c1 * g1), h[1]))
        v1 = np.float32(sr16(fma32(b2, vf, c2 * (g1 * g1)), h[2]))
        q = m1 / (np.sqrt(v1) + eps)
        w1 = sr16(fma32(-alpha, q, wf), h[3])
        assert val(ow[i]) == w1 and val(om[i]) == m1 and val(ov[i]) == v1, i
        assert o8[i] == oracle.fp8_quantize(np.float32([w1]))[0]


def test_first_step_is_lr_times_sign():
    rng = np.random.default_rng(951)
    n = 2000
    w = _p16(rng.standard_normal(n) * 0.5)
    g = _p16(rng.standard_normal(n) * 1e-2)
    zeros = np.zeros(n, np.uint16)
    lr = 2.0 ** -7
    ow, _, _, _ = oracle.adam_update(w, g, zeros, zeros, lr=lr, t=1, seed=4)
    d = oracle.p16_value(ow) - oracle.p16_value(w)
    gv = oracle.p16_value(g)
    # gradients whose square stays well inside FP16's range (v = 0.001 g^2)
    big = np.abs(gv) >= 4e-3
    assert big.sum() > n // 2
    sgn = np.sign(gv)
    # within the FP16 rounding of the moments, the division and the update
    step_err = 3 * 2.0 ** -9 * lr + np.abs(oracle.p16_value(w)) * 2.0 ** -9
    assert np.all(np.abs(d + lr * sgn)[big] <= step_err[big])


def test_stochastic_rounding_keeps_tiny_updates():
    """w = 1, every update 1/8 of a P16 step (2^-12): nearest rounding drops
    it, stochastic rounding moves w by that amount on average."""
    n = 8192
    w = _p16(np.ones(n))
    g = _p16(np.full(n, 1e-3))
    m = _p16(np.full(n, 1e-3))       # with g: m' stays 1e-3 up to rounding
    v = _p16(np.full(n, 1e-6))       # v' ~ 1e-6: m / sqrt(v) ~ 1
    alpha_target = 2.0 ** -12
    lr = alpha_target * (1 - 0.9) / math.sqrt(1 - 0.999)      # t = 1
    ow, om, ov, _ = oracle.adam_update(w, g, m, v, lr=lr, t=1, seed=9)
    q = oracle.p16_value(om) / (np.sqrt(oracle.p16_value(ov)) + 1e-8)
    expect = 1.0 - oracle.adam_step_size(lr, 0.9, 0.999, 1) * q
    got = oracle.p16_value(ow)
    assert set(np.unique(got)) <= {1.0, 1.0 - 2.0 ** -10, 1.0 - 2.0 ** -9}
    sigma = 2.0 ** -10 / math.sqrt(n)
    assert abs(float(np.mean(got)) - float(np.mean(expect))) < 5 * sigma
    assert float(np.mean(got)) < 1.0 - 2.0 ** -13          # moved by ~2^-12


def test_trajectory_follows_float64_adam():
    rng = np.random.default_rng(952)
    n, steps = 4096, 20
    w0 = rng.standard_normal(n) * 0.1
    # gradients bounded away from zero: 0.001 g^2 stays far inside FP16's
    # range (a second moment that underflows would make m / sqrt(v) blow up
    # in any precision that flushes it)
    z = rng.standard_normal((steps, n))
    G = np.sign(z) * (0.5 + np.abs(z)) * 1e-2
    lr, b1, b2, eps = 1e-3, 0.9, 0.999, 1e-8
    w, m, v = _p16(w0), np.zeros(n, np.uint16), np.zeros(n, np.uint16)
    wd, md, vd = w0.copy(), np.zeros(n), np.zeros(n)
    for t in range(1, steps + 1):
        w, m, v, _ = oracle.adam_update(w, _p16(G[t - 1]), m, v, lr=lr, t=t, seed=1, offset=t)
        gd = oracle.p16_value(_p16(G[t - 1]))
        md = b1 * md + (1 - b1) * gd
        vd = b2 * vd + (1 - b2) * gd * gd
        wd = wd - lr * (md / (1 - b1 ** t)) / (np.sqrt(vd / (1 - b2 ** t)) + eps)
    moved = wd - w0
    err = oracle.p16_value(w) - wd
    # FP16 master weights hold ~2^-10 relative precision; the drift is SR noise
    assert np.sqrt(np.mean(err ** 2)) < 0.05 * np.sqrt(np.mean(moved ** 2))
    assert abs(float(np.mean(err))) < 0.01 * np.sqrt(np.mean(moved ** 2))


def test_argument_checks():
    z = np.zeros(4, np.uint16)
    with pytest.raises(ValueError):
        oracle.adam_update(z, z, z, z, lr=1e-3, t=0)
