"""Pins for the oracle's training step of a fully connected network
(oracle/mlp.py):

* ReLU on codes is ReLU on values, over every FP8 and FP16 code;
* the loss gradient and the ReLU backward on hand-worked values;
* with lr = 0, weight decay 0 and momentum 0 the step leaves the weights
  unchanged and leaves each layer's loss-scaled weight gradient in its
  momentum buffer: that gradient follows float64 backpropagation of the same
  network (within the formats' rounding), which pins the chain's structure
  (transposes, masks, loss scaling, the FP16 last layer).
"""
import numpy as np

import oracle
from oracle import mlp


def test_relu_codes_every_code():
    c8 = np.arange(256, dtype=np.uint8)
    v = oracle.p8_value(c8)
    r = oracle.p8_value(mlp.relu8(c8))
    nan = np.isnan(v)
    assert np.all(np.isnan(r[nan]))
    assert np.array_equal(r[~nan], np.maximum(v[~nan], 0.0))
    assert np.all(mlp.relu8(c8)[nan] == 0x7F)
    c16 = np.arange(65536, dtype=np.uint16)
    v = oracle.p16_value(c16)
    r = oracle.p16_value(mlp.relu16(c16))
    nan = np.isnan(v)
    assert np.all(np.isnan(r[nan])) and np.all(mlp.relu16(c16)[nan] == 0x7F00)
    assert np.array_equal(r[~nan], np.maximum(v[~nan], 0.0))
    # ReLU commutes with rounding to FP8
    z = oracle.fp16_quantize(np.linspace(-3, 3, 1001).astype(np.float32))
    assert np.array_equal(mlp.relu8(oracle.fp8_quantize(z)), oracle.fp8_quantize(mlp.relu16(z)))


def test_loss_gradient_and_relu_backward_values():
    y = oracle.fp16_quantize(np.float32([1.5, -2.0, 0.25, 3.0]))
    t = oracle.fp16_quantize(np.float32([1.0, 1.0, 0.25, -1.0]))
    e = oracle.p16_value(mlp.mse_grad_fp16(y, t, np.float32(1000.0 / 256.0)))
    assert list(e) == [0.5 * 3.90625, -3.0 * 3.90625, 0.0, 4.0 * 3.90625]
    d = oracle.fp16_quantize(np.float32([1.0, 2.0, -3.0, 0.1]))
    z = oracle.fp16_quantize(np.float32([0.5, -0.5, 0.0, 2.0]))
    got = oracle.p8_value(mlp.relu_backward_fp8(d, z))
    assert list(got) == [1.0, 0.0, 0.0, float(oracle.p8_value(oracle.fp8_quantize(np.float32([0.1])))[0])]


def test_zero_rate_step_stores_backprop_gradients():
    rng = np.random.default_rng(990)
    widths = (40, 24, 16, 12)
    B = 32
    x = rng.standard_normal((B, widths[0])).astype(np.float32)
    X8 = oracle.fp8_quantize(x)
    T16 = oracle.fp16_quantize(rng.standard_normal((B, widths[-1])).astype(np.float32))
    W16 = [oracle.fp16_quantize((rng.standard_normal((widths[l], widths[l + 1])) /
                                 np.sqrt(widths[l])).astype(np.float32))
           for l in range(len(widths) - 1)]
    V16 = [np.zeros_like(w) for w in W16]
    scale = 1000.0
    Wn, Vn, W8n, Y = mlp.mlp_step(widths, X8, T16, W16, V16, lr=0.0, momentum=0.0,
                                  weight_decay=0.0, loss_scale=scale, seed=1, t=0)
    for a, b in zip(Wn, W16):
        assert np.array_equal(a, b)
    # float64 backpropagation of the same network with the same quantization
    # points (FP8 activations, errors and hidden weights; FP16 last layer and
    # loss gradient), loss 1/(2B) sum (y - t)^2, times the scale
    q8 = lambda x: oracle.p8_value(oracle.fp8_quantize(np.asarray(x, np.float32)))
    q16 = lambda x: oracle.p16_value(oracle.fp16_quantize(np.asarray(x, np.float32)))
    L = len(widths) - 1
    Wv = [q8(oracle.p16_value(W16[l])) for l in range(L - 1)]
    Wv.append(oracle.p16_value(W16[L - 1]))
    A = [oracle.p8_value(X8)]
    Zs = []
    for l in range(L):
        z = A[-1] @ Wv[l]
        Zs.append(z)
        relu = np.maximum(z, 0.0)
        A.append(q16(relu) if l == L - 2 else q8(relu))
    y = Zs[-1]
    # (an FP8 activation next to a rounding boundary may round the other way,
    # so the comparison is in norm)
    assert np.linalg.norm(oracle.p16_value(Y) - y) / np.linalg.norm(y) < 0.05
    g = q16((oracle.p16_value(Y) - oracle.p16_value(T16)) * scale / B)
    grads = [None] * L
    for l in range(L - 1, -1, -1):
        grads[l] = A[l].T @ g
        if l > 0:
            g = q8((g @ Wv[l].T) * (Zs[l - 1] > 0))
    for l in range(L):
        got = oracle.p16_value(Vn[l])
        err = np.linalg.norm(got - grads[l]) / np.linalg.norm(grads[l])
        assert err < 0.05, (l, err)
