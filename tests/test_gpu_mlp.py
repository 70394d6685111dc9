"""GPU parity of the element-wise steps and of whole training steps of a
fully connected network (paper_1812_08011_amd.mlp) with the oracle's step
(oracle/mlp.py), bit for bit: weights, momentum buffers, FP8 weight copies
and outputs, for a small network over two steps and for the speech DNN
(440 -> 1024 x 5 -> 6000, batch 256) over one step."""
import numpy as np
import pytest
import torch

import oracle
import paper_1812_08011_amd as fp8t
import workloads
from oracle import mlp as omlp
from paper_1812_08011_amd.mlp import Fp8Mlp
from tests.gpu_util import DEV, dev, host, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fp8t.lib()
    yield


def test_relu_codes_every_code():
    c8 = np.arange(256, dtype=np.uint8)
    c16 = np.arange(65536, dtype=np.uint16)
    say("relu_codes fp8 / fp16, every code")
    y8 = torch.empty(256, dtype=torch.uint8, device=DEV)
    fp8t.relu_codes(dev(c8), 8, y8, 256)
    assert np.array_equal(host(y8), omlp.relu8(c8))
    x16 = dev(c16)
    fp8t.relu_codes(x16, 16, x16, 65536)                      # in place
    assert np.array_equal(host(x16), omlp.relu16(c16))


def test_relu_backward_and_loss_gradient():
    rng = np.random.default_rng(991)
    n = 100_003
    d = oracle.fp16_quantize((rng.standard_normal(n) * 30).astype(np.float32))
    z = oracle.fp16_quantize(rng.standard_normal(n).astype(np.float32))
    y = oracle.fp16_quantize((rng.standard_normal(n) * 2).astype(np.float32))
    specials = np.uint16([0x0000, 0x8000, 0x7E00, 0xFE00, 0x7F00, 0x0001, 0x7DFF, 0xFDFF])
    for a in (d, z, y):
        idx = rng.choice(n, n // 100, replace=False)
        a[idx] = rng.choice(specials, idx.size)
    e8 = torch.empty(n, dtype=torch.uint8, device=DEV)
    for scale in (1.0, 1000.0):
        say(f"relu_backward_fp8 scale={scale}")
        fp8t.relu_backward_fp8(dev(d), dev(z), e8, n, scale)
        assert np.array_equal(host(e8), omlp.relu_backward_fp8(d, z, scale))
    e16 = torch.empty(n, dtype=torch.uint16, device=DEV)
    for s in (np.float32(1000.0) / np.float32(256.0), np.float32(3e-9), np.float32(1e30)):
        say(f"mse_grad_fp16 scale={s}")
        fp8t.mse_grad_fp16(dev(y), dev(z), e16, n, float(s))
        assert np.array_equal(host(e16), omlp.mse_grad_fp16(y, z, s))


def run_steps(widths, batch, steps, seed):
    d = workloads.speech_mlp(seed=seed, batch=batch, widths=widths)
    X8 = oracle.fp8_quantize(d["X"])
    T16 = oracle.fp16_quantize(d["T"])
    W16 = [oracle.fp16_quantize(w) for w in d["W"]]
    V16 = [np.zeros_like(w) for w in W16]
    net = Fp8Mlp(widths, batch)
    net.set_weights(W16)
    Xd, Td = dev(X8), dev(T16)
    hp = dict(lr=d["lr"], momentum=d["momentum"], weight_decay=d["weight_decay"],
              loss_scale=d["loss_scale"], seed=d["seed"])
    for t in range(steps):
        say(f"mlp step {t} widths={widths} batch={batch}")
        Yg = host(net.step(Xd, Td, t=t, **hp))
        W16, V16, W8, Yo = omlp.mlp_step(widths, X8, T16, W16, V16, t=t, **hp)
        assert np.array_equal(Yg, Yo), ("Y", t)
        for l in range(len(widths) - 1):
            assert np.array_equal(host(net.W16[l]), W16[l]), ("W16", t, l)
            assert np.array_equal(host(net.V16[l]), V16[l]), ("V16", t, l)
            if l < len(widths) - 2:
                assert np.array_equal(host(net.W8[l]), W8[l]), ("W8", t, l)


def test_small_network_two_steps():
    run_steps((440, 64, 48, 96), 32, 2, seed=7)


def test_speech_dnn_step():
    run_steps(workloads.SPEECH_LAYERS[0][:1] + tuple(fo for _, fo in workloads.SPEECH_LAYERS),
              256, 1, seed=6)
