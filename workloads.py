"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic (no rounding into FP8 or FP16, no accumulation).  Both the
CPU oracle and the GPU path take their inputs from here and quantize them with
their own code.  Every array is drawn with ``numpy.random.default_rng(seed)``
(PCG64) in float64 and converted to float32; that float32 array is the
canonical input.  Scales (the loss scale, the 2^-2 of the small GEMM) are not
applied here: they are passed to the quantizer, which multiplies in FP32.

Workloads (the paper's datasets and trained weights are not available, so the
shapes and value distributions stand in for them):

* ``small``   -- one 128x128x1024 GEMM and a 4096-element weight update.
* ``conv``    -- a 3x3 convolution of a 50-layer residual CNN stage lowered to
  GEMMs (Sec. 2.2 lowers convolutions to GEMMs): batch 256, 14x14, 256 -> 256
  channels, giving forward 50176x256x2304, backward-data 50176x2304x256 and
  weight-gradient 2304x256x50176 (ImageNet-ResNet50 stand-in, Table 1).
* ``sweep``   -- weight-gradient-like 512x512xK GEMMs with long K and 1%
  outliers (the long-accumulation study of Sec. 4.2).
* ``speech``  -- the six fully connected layers of the BN50 speech DNN
  (Appendix A) at batch 256 (BN50 stand-in, Table 1).
* ``update``  -- a 25.6M-parameter SGD update (ResNet50 parameter count).
"""
import numpy as np


def _normal(rng, shape, std=1.0):
    return (rng.standard_normal(shape) * std).astype(np.float32)


# ---- small GEMM + small update ---------------------------------------------

def small_gemm(seed=0, M=128, N=128, K=1024):
    """A (MxK) and B (KxN) from N(0,1); quantizer scale 2^-2."""
    rng = np.random.default_rng(seed)
    A = _normal(rng, (M, K))
    B = _normal(rng, (K, N))
    return A, B, 0.25


def small_update(seed=1, n=4096):
    """Weights N(0, 0.05), gradients N(0, 1e-3); lr 0.1, no momentum."""
    rng = np.random.default_rng(seed)
    w = _normal(rng, (n,), 0.05)
    g = _normal(rng, (n,), 1e-3)
    return dict(w=w, g=g, v=None, lr=0.1, momentum=0.0, weight_decay=0.0,
                seed=1, offset=0)


# ---- conv stage lowered to GEMMs --------------------------------------------

CONV = dict(batch=256, hw=14, cin=256, cout=256, kh=3, kw=3)


def im2col_3x3(X):
    """NHWC input -> (N*H*W) x (3*3*C) columns, stride 1, zero padding 1,
    column order (kh, kw, cin)."""
    n, h, w, c = X.shape
    Xp = np.zeros((n, h + 2, w + 2, c), dtype=X.dtype)
    Xp[:, 1:h + 1, 1:w + 1, :] = X
    cols = np.empty((n * h * w, 9 * c), dtype=X.dtype)
    for a in range(3):
        for b in range(3):
            t = a * 3 + b
            cols[:, t * c:(t + 1) * c] = Xp[:, a:a + h, b:b + w, :].reshape(n * h * w, c)
    return cols


def conv_stage_input(seed=2, batch=256, hw=14, cin=256, cout=256):
    """The conv stage before lowering: X NHWC ~ ReLU(N(0,1)), W (9 cin x cout)
    ~ N(0, sqrt(2/K)) in (kh, kw, cin) row order, dY (batch hw hw x cout) ~
    N(0, 1e-3) with a loss scale of 1024 applied by the quantizer -- the same
    draws as conv_gemms."""
    rng = np.random.default_rng(seed)
    X = np.maximum(rng.standard_normal((batch, hw, hw, cin)), 0.0).astype(np.float32)
    K = 9 * cin
    W = _normal(rng, (K, cout), np.sqrt(2.0 / K))
    dY = _normal(rng, (batch * hw * hw, cout), 1e-3)
    return dict(X=X, W=W, dY=dY, dy_scale=1024.0)


def conv_gemms(seed=2, batch=256, hw=14, cin=256, cout=256):
    """Returns dict with Xcol (M x K), W (K x cout), dY (M x cout) as float32
    and the loss scale for dY.

    X ~ ReLU(N(0,1)) (post-ReLU activations: half exact zeros, half-normal
    tail), W ~ N(0, sqrt(2/K)) (He initialisation), dY ~ N(0, 1e-3) times a
    loss scale of 1024 applied by the quantizer."""
    rng = np.random.default_rng(seed)
    X = np.maximum(rng.standard_normal((batch, hw, hw, cin)), 0.0).astype(np.float32)
    Xcol = im2col_3x3(X)
    K = 9 * cin
    W = _normal(rng, (K, cout), np.sqrt(2.0 / K))
    dY = _normal(rng, (batch * hw * hw, cout), 1e-3)
    return dict(Xcol=Xcol, W=W, dY=dY, dy_scale=1024.0)


# ---- long-accumulation sweep -------------------------------------------------

SWEEP_K = (4096, 16384, 65536)


def sweep_gemm(K, seed=3, M=512, N=512):
    """A stored K x M (weight-gradient layout, op(A) = A^T) and B stored K x N,
    N(0,1) with a 1% Bernoulli mask of outliers scaled by 16."""
    rng = np.random.default_rng(seed)
    out = []
    for cols in (M, N):
        z = rng.standard_normal((K, cols))
        mask = rng.random((K, cols)) < 0.01
        z[mask] *= 16.0
        out.append(z.astype(np.float32))
    return out[0], out[1]


def accumulation_vector(n, seed=11):
    """Sec. 2.3, Fig. 3(b): a vector drawn from a uniform distribution with
    mean 1 and standard deviation 1, i.e. U(1 - sqrt(3), 1 + sqrt(3))."""
    rng = np.random.default_rng(seed)
    r3 = np.sqrt(3.0)
    return rng.uniform(1.0 - r3, 1.0 + r3, size=n).astype(np.float32)


# ---- speech DNN layers ---------------------------------------------------------

SPEECH_LAYERS = ((440, 1024), (1024, 1024), (1024, 1024), (1024, 1024),
                 (1024, 1024), (1024, 6000))


def speech_layer(l, seed=4, batch=256):
    """Layer l of the BN50 DNN: X (batch x fan_in) ~ N(0,1),
    W (fan_in x fan_out) ~ N(0, 1/sqrt(fan_in)), E (batch x fan_out) ~
    N(0, 1e-3) with a loss scale of 1000 applied by the quantizer.  Inputs of
    different layers are independent draws."""
    rng = np.random.default_rng([seed, l])
    fi, fo = SPEECH_LAYERS[l]
    X = _normal(rng, (batch, fi))
    W = _normal(rng, (fi, fo), 1.0 / np.sqrt(fi))
    E = _normal(rng, (batch, fo), 1e-3)
    return dict(X=X, W=W, E=E, e_scale=1000.0)


def speech_mlp(seed=6, batch=256, widths=(440, 1024, 1024, 1024, 1024, 1024, 6000)):
    """A whole training step of the DNN on synthetic regression data: input X
    (batch x widths[0]) ~ N(0,1), targets T (batch x widths[-1]) ~ N(0,1),
    weights W_l (widths[l] x widths[l+1]) ~ N(0, 1/sqrt(fan_in)); SGD with
    lr 0.003, momentum 0.9, weight decay 1e-4, loss scale 1000 (the loss is
    the squared error summed over the 6000 outputs and averaged over the
    batch; in float32, lr 0.03 and above diverges within a few steps on this
    data, lr 0.003 lowers the loss steadily)."""
    rng = np.random.default_rng(seed)
    X = _normal(rng, (batch, widths[0]))
    T = _normal(rng, (batch, widths[-1]))
    W = [_normal(rng, (widths[l], widths[l + 1]), 1.0 / np.sqrt(widths[l]))
         for l in range(len(widths) - 1)]
    return dict(X=X, T=T, W=W, lr=0.003, momentum=0.9, weight_decay=1e-4, loss_scale=1000.0,
                seed=21)


# ---- big weight update -----------------------------------------------------------

def big_update(seed=5, n=25_600_000):
    """Weights N(0, 0.02), gradients and momentum N(0, 1e-4); lr 0.1,
    momentum 0.9, weight decay 1e-4, Philox seed 7."""
    rng = np.random.default_rng(seed)
    w = _normal(rng, (n,), 0.02)
    g = _normal(rng, (n,), 1e-4)
    v = _normal(rng, (n,), 1e-4)
    return dict(w=w, g=g, v=v, lr=0.1, momentum=0.9, weight_decay=1e-4,
                seed=7, offset=0)
