"""Seeded synthetic layer inputs shaped like the paper's workloads.

This module only draws random tensors; it holds none of the quantizer or
contraction arithmetic and imports nothing else from the package, so the
tests can hand the same inputs to the HIP path and to the CPU oracle.

All draws use numpy ``Generator(PCG64(seed))`` in the order X, W, G, in
float64, rounded to float32.  The gradient rows are heavy-tailed across
samples, which is what motivates the per-sample and block Householder
quantizers (Sec. 4.1: near-zero gradients for well-classified samples, a few
large outlier rows).
"""
import numpy as np


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def lognormal_row_gradient(rng, n, d, sigma=2.0):
    """Rows s_i * N(0, 1) with s_i ~ LogNormal(0, sigma)."""
    s = rng.lognormal(0.0, sigma, size=(n, 1))
    return (s * rng.standard_normal((n, d))).astype(np.float32)


def linear_small(seed=0, n=128, d_in=256, d_out=256):
    """Linear layer 128 x 256 -> 256: X = ReLU(N(0,1)), W ~ N(0, 2/d_in), log-normal row scales."""
    rng = _rng(seed)
    X = np.maximum(rng.standard_normal((n, d_in)), 0.0).astype(np.float32)
    W = (rng.standard_normal((d_out, d_in)) * np.sqrt(2.0 / d_in)).astype(np.float32)
    G = lognormal_row_gradient(rng, n, d_out)
    return X, W, G


def mlp(seed=0, n=64, widths=(24, 32, 32, 16)):
    """ReLU MLP inputs: X ~ N(0,1) [n, widths[0]]; W_i ~ N(0, 2/widths[i]) [widths[i+1], widths[i]]
    (He); top output gradient G with log-normal row scales [n, widths[-1]]."""
    rng = _rng(seed)
    X = rng.standard_normal((n, widths[0])).astype(np.float32)
    Ws = [(rng.standard_normal((widths[i + 1], widths[i])) * np.sqrt(2.0 / widths[i])).astype(np.float32)
          for i in range(len(widths) - 1)]
    G = lognormal_row_gradient(rng, n, widths[-1])
    return X, Ws, G


def linear_outlier(seed=0, n=8192, d_in=1024, d_out=4096, frac=0.01, big=10.0, small=0.01):
    """Transformer-FFN shaped layer: X ~ N(0,1), W ~ N(0, 1/d_in), G with 1% outlier rows.

    round(frac * n) rows, chosen without replacement, are big * N(0,1); the
    rest are small * N(0,1).
    """
    rng = _rng(seed)
    X = rng.standard_normal((n, d_in)).astype(np.float32)
    W = (rng.standard_normal((d_out, d_in)) * np.sqrt(1.0 / d_in)).astype(np.float32)
    n_out = int(round(frac * n))
    rows = rng.choice(n, size=n_out, replace=False)
    scale = np.full((n, 1), small)
    scale[rows] = big
    G = (scale * rng.standard_normal((n, d_out))).astype(np.float32)
    return X, W, G


def linear_single_outlier(seed=0, n=4096, d_in=4096, d_out=4096, factor=1000.0):
    """Square layer with G ~ N(0,1) except one row (drawn from the seed) scaled by `factor`."""
    rng = _rng(seed)
    X = rng.standard_normal((n, d_in)).astype(np.float32)
    W = (rng.standard_normal((d_out, d_in)) * np.sqrt(1.0 / d_in)).astype(np.float32)
    G = rng.standard_normal((n, d_out))
    G[int(rng.integers(n))] *= factor
    return X, W, G.astype(np.float32)


def conv_layer(seed=0, n=128, c=64, h=56, w=56, o=64, k=3, stride=1, pad=1, stem=False):
    """Conv layer in NHWC: X post-ReLU half-normal (N(0,1) for a stem input),
    W He-init N(0, 2/fan_in) as [o, k, k, c], G per-sample LogNormal(0, 2) scales."""
    rng = _rng(seed)
    X = rng.standard_normal((n, h, w, c))
    if not stem:
        X = np.maximum(X, 0.0)
    X = X.astype(np.float32)
    W = (rng.standard_normal((o, k, k, c)) * np.sqrt(2.0 / (k * k * c))).astype(np.float32)
    ho = (h + 2 * pad - k) // stride + 1
    wo = (w + 2 * pad - k) // stride + 1
    G = lognormal_row_gradient(rng, n, ho * wo * o).reshape(n, ho, wo, o)
    return X, W, G


# ResNet-50 v1.5 conv shapes (224 x 224 input): (c_in, c_out, k, stride, h_in, count)
RESNET50_CONVS = [
    (3, 64, 7, 2, 224, 1),
    (64, 64, 1, 1, 56, 1), (64, 64, 3, 1, 56, 3), (64, 256, 1, 1, 56, 4),
    (256, 64, 1, 1, 56, 2), (256, 128, 1, 1, 56, 1),
    (128, 128, 3, 2, 56, 1), (128, 512, 1, 1, 28, 4), (256, 512, 1, 2, 56, 1),
    (512, 128, 1, 1, 28, 3), (128, 128, 3, 1, 28, 3), (512, 256, 1, 1, 28, 1),
    (256, 256, 3, 2, 28, 1), (256, 1024, 1, 1, 14, 6), (512, 1024, 1, 2, 28, 1),
    (1024, 256, 1, 1, 14, 5), (256, 256, 3, 1, 14, 5), (1024, 512, 1, 1, 14, 1),
    (512, 512, 3, 2, 14, 1), (512, 2048, 1, 1, 7, 3), (1024, 2048, 1, 2, 14, 1),
    (2048, 512, 1, 1, 7, 2), (512, 512, 3, 1, 7, 2),
]
