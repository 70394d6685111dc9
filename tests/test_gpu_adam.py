"""GPU parity of adam_update (ADAM in FP16 with stochastic rounding) with the
oracle, bit for bit: sizes with ragged ends, with and without the FP8 copy,
step numbers from 1 to 10^6, 64-bit seeds and offsets, special codes,
misaligned pointers, and the 25.6 M-parameter size of a 50-layer residual
CNN."""
import numpy as np
import pytest
import torch

import oracle
import paper_1812_08011_amd as fp8t
from tests.gpu_util import DEV, dev, host, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fp8t.lib()
    yield


def _p16(x):
    return oracle.fp16_quantize(np.asarray(x, np.float32))


def _state(rng, n):
    w = _p16(rng.standard_normal(n) * 0.05)
    g = _p16(rng.standard_normal(n) * 1e-2)
    m = _p16(rng.standard_normal(n) * 1e-3)
    v = _p16(np.abs(rng.standard_normal(n)) * 1e-5)
    return w, g, m, v


def _case(w, g, m, v, with_w8=True, lr=1e-3, b1=0.9, b2=0.999, eps=1e-8, wd=1e-4, t=3,
          seed=5, offset=0):
    n = w.size
    wd_, gd, md, vd = dev(w), dev(g), dev(m), dev(v)
    w8 = torch.zeros(n, dtype=torch.uint8, device=DEV) if with_w8 else None
    say(f"adam_update n={n} w8={with_w8} lr={lr} b1={b1} b2={b2} eps={eps} wd={wd} t={t} "
        f"seed={seed} offset={offset}")
    fp8t.adam_update(wd_, gd, md, vd, w8, n, lr, b1, b2, eps, wd, t, seed, offset)
    ow, om, ov, o8 = oracle.adam_update(w, g, m, v, lr=lr, beta1=b1, beta2=b2, eps=eps,
                                        weight_decay=wd, t=t, seed=seed, offset=offset,
                                        want_w8=with_w8)
    assert np.array_equal(host(wd_), ow)
    assert np.array_equal(host(md), om)
    assert np.array_equal(host(vd), ov)
    if with_w8:
        assert np.array_equal(host(w8), o8)


def test_adam_variants():
    rng = np.random.default_rng(960)
    for n in (1, 2, 3, 4097, 100_001):
        for with_w8 in (True, False):
            _case(*_state(rng, n), with_w8=with_w8)
    for t in (1, 10, 10 ** 6):
        _case(*_state(rng, 20_000), t=t)
    _case(*_state(rng, 20_000), seed=2 ** 63 + 7, offset=2 ** 40 + 3)
    _case(*_state(rng, 20_000), b1=0.5, b2=0.9, eps=1e-4, wd=0.0, lr=0.1)


@pytest.mark.parametrize("n", [20_001, 4_500_003])
def test_adam_specials(n):
    """Special codes among ordinary values: their pairs take the general
    path, the others the normal-range one (at the larger size every thread of
    the capped grid loops over several pairs)."""
    rng = np.random.default_rng(961)
    w, g, m, v = _state(rng, n)
    specials = np.uint16([0x0000, 0x8000, 0x0001, 0x81FF, 0x7DFF, 0xFDFF, 0x7E00, 0xFE00,
                          0x7F00, 0xBE00])                     # 0xBE00: -1 (negative v)
    for a in (w, g, m, v):
        idx = rng.choice(n, size=n // 50, replace=False)
        a[idx] = rng.choice(specials, size=idx.size)
    _case(w, g, m, v)
    _case(w, g, m, v, eps=0.0, lr=1.0)


def test_adam_misaligned():
    rng = np.random.default_rng(962)
    n = 10_001
    w, g, m, v = _state(rng, n + 1)
    wd_, gd, md, vd = dev(w), dev(g), dev(m), dev(v)
    w8 = torch.zeros(n + 1, dtype=torch.uint8, device=DEV)
    say("adam_update misaligned")
    fp8t.lib().adam_update(wd_.data_ptr() + 2, gd.data_ptr() + 2, md.data_ptr() + 2,
                           vd.data_ptr() + 2, w8.data_ptr() + 1, n, 1e-3, 0.9, 0.999, 1e-8,
                           0.0, 2, 3, 4, torch.cuda.current_stream().cuda_stream)
    ow, om, ov, o8 = oracle.adam_update(w[1:], g[1:], m[1:], v[1:], lr=1e-3, t=2, seed=3,
                                        offset=4)
    assert np.array_equal(host(wd_)[1:], ow) and np.array_equal(host(md)[1:], om)
    assert np.array_equal(host(vd)[1:], ov) and np.array_equal(host(w8)[1:], o8)


def test_adam_full_size():
    rng = np.random.default_rng(963)
    _case(*_state(rng, 25_600_000), t=100, seed=7)
