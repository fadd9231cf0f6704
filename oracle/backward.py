"""FQT layer backward (oracle; test infrastructure only).

Sec. 2.2, Eq. (linear-sq-backprop), with the gradient bifurcation of App. E:

    grad_W = Q_b1(G)^T Q_f(X)        (Q_b1: 8-bit stochastic PTQ)
    grad_X = Q_b2(G)   Q_theta(W)    (Q_b2: PTQ, PSQ or BHQ, 4-8 bits)

in PyTorch orientation: X [N, d_in], W [d_out, d_in], G = dL/dY [N, d_out].
The paper writes Theta [D_in, D_out] and the transposed products (Sec. 2.1).
Q_f and Q_theta are deterministic 8-bit PTQ (App. E).

Two results are produced:
  * the exact integer accumulators of the offset codes (int64 matmul), which
    the int8 contractions must reproduce bit for bit;
  * the dequantized gradients: a float64 matmul of the real values each
    quantizer represents, rounded once to float32.

Conv layers (``conv_backward``) are the same products over an explicit im2col
of the NHWC tensors (rows = samples for the gradient quantizer, Sec. 4.1).
"""
import numpy as np

from . import quantizers as Q


def quantize_gradient(G, spec, seed, stream):
    kind, bits, k = spec
    if kind == "ptq":
        return Q.quantize_ptq(G, bits, True, seed, stream)
    if kind == "psq":
        return Q.quantize_psq(G, bits, seed, stream)
    if kind == "bhq":
        return Q.quantize_bhq(G, bits, k, seed, stream)
    if kind == "shift":
        return Q.quantize_shift(G, bits, seed, stream)
    raise ValueError(kind)


def slot_codes(q):
    """Offset codes in the row order the contraction consumes (slot order for BHQ)."""
    return Q.offset_codes(q)


def linear_backward(X, W, G, qb_x=("psq", 8, 0), qb_w=("ptq", 8, 0), f_bits=8, theta_bits=8, seed=0):
    """One linear layer's FQT backward.  Returns a dict of every intermediate."""
    X = np.asarray(X, np.float32)
    W = np.asarray(W, np.float32)
    G = np.asarray(G, np.float32)
    qx = Q.quantize_ptq(X, f_bits, False)
    qw = Q.quantize_ptq(W, theta_bits, False)
    qb1 = quantize_gradient(G, qb_w, seed, 0)
    qb2 = quantize_gradient(G, qb_x, seed, 1)
    Xr, Wr = Q.dequantize(qx), Q.dequantize(qw)
    G1r, G2r = Q.dequantize(qb1), Q.dequantize(qb2)
    grad_W = (G1r.T @ Xr).astype(np.float32)
    grad_X = (G2r @ Wr).astype(np.float32)
    acc_w = (Q.shifted_codes(qb1) if qb1["kind"] == "shift" else Q.offset_codes(qb1)).T @ Q.offset_codes(qx)
    acc_x = slot_codes(qb2) @ Q.offset_codes(qw)
    return dict(qx=qx, qw=qw, qb1=qb1, qb2=qb2, grad_W=grad_W, grad_X=grad_X,
                acc_w=acc_w, acc_x=acc_x, grad_W64=G1r.T @ Xr, grad_X64=G2r @ Wr)


# ----------------------------------------------------------------------------
# conv
# ----------------------------------------------------------------------------

def conv_out_size(h, k, stride, pad):
    return (h + 2 * pad - k) // stride + 1


def im2col(x, kh, kw, stride, pad, ho, wo):
    """Rows (n, y, x) of output pixels, columns (r, s, c) of taps; zeros outside."""
    n, h, w, c = x.shape
    cols = np.zeros((n, ho, wo, kh, kw, c), x.dtype)
    for r in range(kh):
        for s in range(kw):
            for oy in range(ho):
                iy = oy * stride - pad + r
                if iy < 0 or iy >= h:
                    continue
                for ox in range(wo):
                    ix = ox * stride - pad + s
                    if 0 <= ix < w:
                        cols[:, oy, ox, r, s, :] = x[:, iy, ix, :]
    return cols.reshape(n * ho * wo, kh * kw * c)


def col2im(cols, n, h, w, c, kh, kw, stride, pad, ho, wo):
    """Adjoint of im2col: scatter-add tap columns back onto input pixels."""
    cols = cols.reshape(n, ho, wo, kh, kw, c)
    out = np.zeros((n, h, w, c), cols.dtype)
    for r in range(kh):
        for s in range(kw):
            for oy in range(ho):
                iy = oy * stride - pad + r
                if iy < 0 or iy >= h:
                    continue
                for ox in range(wo):
                    ix = ox * stride - pad + s
                    if 0 <= ix < w:
                        out[:, iy, ix, :] += cols[:, oy, ox, r, s, :]
    return out


def conv_backward(X, W, G, stride, pad, qb_x=("bhq", 5, 64), qb_w=("ptq", 8, 0),
                  f_bits=8, theta_bits=8, seed=0):
    """FQT backward of a conv layer, NHWC X [n,h,w,c], W [o,kh,kw,c], G [n,ho,wo,o].

    The forward conv is Y = im2col(X) W^T; its linear-layer backward (Sec. 2.1)
    is grad_W = G^T im2col(X) and grad_X = col2im(G W).  Quantizers act on the
    NHWC tensors with rows = samples (Sec. 4.1): X and W per tensor, G per
    sample / per group of samples.  Padding contributes exact zeros.
    """
    X = np.asarray(X, np.float32)
    W = np.asarray(W, np.float32)
    G = np.asarray(G, np.float32)
    n, h, w, c = X.shape
    o, kh, kw, _ = W.shape
    ho, wo = G.shape[1], G.shape[2]
    qx = Q.quantize_ptq(X.reshape(n, -1), f_bits, False)
    qw = Q.quantize_ptq(W.reshape(o, -1), theta_bits, False)
    qb1 = quantize_gradient(G.reshape(n, -1), qb_w, seed, 0)
    qb2 = quantize_gradient(G.reshape(n, -1), qb_x, seed, 1)
    Xr = Q.dequantize(qx).reshape(n, h, w, c)
    Wr = Q.dequantize(qw).reshape(o, kh * kw * c)
    G1r = Q.dequantize(qb1).reshape(n * ho * wo, o)
    G2r = Q.dequantize(qb2).reshape(n * ho * wo, o)
    cols = im2col(Xr, kh, kw, stride, pad, ho, wo)
    grad_W = (G1r.T @ cols)
    grad_X = col2im(G2r @ Wr, n, h, w, c, kh, kw, stride, pad, ho, wo)
    # exact integer accumulators: offset codes, padding taps contribute nothing
    qxo = Q.offset_codes(qx).reshape(n, h, w, c)
    acc_w = Q.offset_codes(qb1).reshape(n * ho * wo, o).T @ im2col(qxo, kh, kw, stride, pad, ho, wo)
    return dict(qx=qx, qw=qw, qb1=qb1, qb2=qb2, grad_W=grad_W.reshape(o, kh, kw, c).astype(np.float32),
                grad_X=grad_X.astype(np.float32), acc_w=acc_w.reshape(o, kh, kw, c),
                grad_W64=grad_W.reshape(o, kh, kw, c), grad_X64=grad_X)
