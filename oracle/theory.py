"""Closed forms of the paper used to pin the oracle (test infrastructure only).

* variance bounds: PTQ, Eq. (variance-scale-shift) / App. C.1; matrix
  quantizer, Eq. (matrix-quantizer-variance) / App. C.2; PSQ, Sec. 4.1 /
  App. C.3; Householder quantizer, Sec. 4.2 / App. C.4;
* the Householder reflection Q = I - 2 n n^T / |n|^2, n = 1/sqrt(k) - e_1
  (Sec. 4.2), as an explicit matrix;
* exact quantizer variance: sum over elements of p (1 - p) (App. C, SR
  variance), mapped through S^-1 (Prop. var, App. B).
"""
import math

import numpy as np

from . import sr
from . import quantizers as Q


def householder_matrix(k):
    """Explicit k x k reflection with normal 1/sqrt(k) * 1 - e_1, float64."""
    n = np.full(k, 1.0 / math.sqrt(k))
    n[0] -= 1.0
    return np.eye(k) - 2.0 * np.outer(n, n) / (n @ n)


def ptq_var_bound(x, bits):
    """N D R^2 / (4 B^2), Eq. (variance-scale-shift)."""
    x = np.asarray(x, np.float64)
    B = Q.n_bins(bits)
    R = x.max() - x.min()
    return x.size * R * R / (4.0 * B * B)


def psq_var_bound(x, bits):
    """D / (4 B^2) * sum_i R_i^2, Sec. 4.1."""
    x = np.asarray(x, np.float64)
    B = Q.n_bins(bits)
    R = x.max(axis=1) - x.min(axis=1)
    return x.shape[1] * float((R * R).sum()) / (4.0 * B * B)


def householder_var_bound(lam1, lam2, k, D, bits):
    """D / (4 B^2) (lam1^(2/3) k^(-1/3) + lam2^(2/3) k^(2/3))^3, Sec. 4.2."""
    B = Q.n_bins(bits)
    return D / (4.0 * B * B) * (lam1 ** (2 / 3) * k ** (-1 / 3) + lam2 ** (2 / 3) * k ** (2 / 3)) ** 3


def inverse_scale_blocks(q):
    """Per group the explicit S^-1 = D^-1 Q block (float64) with its member rows."""
    out = []
    for info in q["plan"]["groups"]:
        base, kg = info["base"], info["size"]
        d = q["scale"][base: base + kg].astype(np.float64)
        Hk = householder_matrix(kg) if kg > 1 else np.eye(1)
        out.append((info, np.diag(1.0 / d) @ Hk))
    return out


def matrix_var_bound(q, D):
    """(D / 4) |S^-1|_F^2, Eq. (matrix-quantizer-variance)."""
    if q["kind"] == "bhq":
        return D / 4.0 * sum(float((Si ** 2).sum()) for _, Si in inverse_scale_blocks(q))
    s = np.asarray(q["scale"], np.float64)
    rows = q["code"].shape[0]
    s = np.broadcast_to(s, (rows,))
    return D / 4.0 * float((1.0 / s ** 2).sum())


def transformed_values(x, q):
    """The float32 values y each code stochastically rounds (slot order for BHQ)."""
    x = np.asarray(x, np.float32)
    if q["kind"] == "ptq":
        return (q["scale"] * (x - q["zero"]).astype(np.float32)).astype(np.float32)
    if q["kind"] in ("psq", "shift"):
        return (q["scale"][:, None] * (x - q["zero"][:, None]).astype(np.float32)).astype(np.float32)
    y = np.zeros_like(x)
    for info in q["plan"]["groups"]:
        info = dict(info, k=q["k"])
        base, kg, mem = info["base"], info["size"], info["members"]
        if kg == 1:
            s, z = q["scale"][base], q["zero"][base]
            y[base] = (s * (x[mem[0]] - z).astype(np.float32)).astype(np.float32)
        else:
            y[base: base + kg] = Q.bhq_transform(x[mem], info)
    return y


def exact_elementwise_variance(x, q):
    """Exact variance of every dequantized element given the inputs, original row order.

    Per element of the code matrix Var = p (1 - p); the dequantized value is
    S^-1 (code + c), so element (i, j) collects sum_p (S^-1)_ip^2 Var[code_pj]
    (Prop. var, App. B).  Ignores the [0, B] clamp, which the range
    construction makes inactive.
    """
    y = transformed_values(x, q)
    v = sr.exact_var_code(y)                     # per code element (slot order for BHQ)
    if q["kind"] == "ptq":
        return v / float(q["scale"]) ** 2
    if q["kind"] in ("psq", "shift"):
        return v / q["scale"][:, None].astype(np.float64) ** 2
    out = np.zeros(v.shape)
    for info, Si in inverse_scale_blocks(q):
        base, kg, mem = info["base"], info["size"], info["members"]
        out[mem] = (Si ** 2) @ v[base: base + kg]
    return out


def exact_quantizer_variance(x, q):
    """Exact total variance of the dequantized result (sum over elements)."""
    return float(exact_elementwise_variance(x, q).sum())


def exact_mean(x, q):
    """E[dequantized result] given the inputs, original row order, float64."""
    y = transformed_values(x, q)
    m = sr.exact_mean_code(y, Q.n_bins(q["bits"]))
    qq = dict(q, code=m)
    if q["kind"] == "bhq":
        return Q.dequantize_bhq(qq)
    return Q.dequantize_affine(qq)
