"""Multi-layer FQT chain on a ReLU MLP (oracle; test infrastructure only).

Layer i (i = 0 .. L-1) of the chain, PyTorch orientation (Sec. 2.1, Eq.
(quantized-forward-propagation)):

    Xt_i = Q_f(A_i),  Wt_i = Q_theta(W_i)       deterministic 8-bit PTQ
    Z_i  = Xt_i Wt_i^T,  A_{i+1} = ReLU(Z_i)     (the last layer is linear)

QAT gradient (Sec. 2.1, Eq. (back-prop); straight-through through Q_f and
Q_theta), with dZ_{L-1} = G the output gradient:

    grad_W_i = dZ_i^T Xt_i,  dA_i = dZ_i Wt_i,  dZ_{i-1} = dA_i * 1[A_i > 0]

FQT gradient (Sec. 2.2, Eq. (quantized-back-prop)): each linear layer's
output gradient dZ_i is quantized, bifurcated as in App. E (Q_b1(dZ_i) for
grad_W_i, Q_b2(dZ_i) for dA_i, independent streams of the layer's seed).  The
ReLU layers apply their Jacobian exactly: their quantizer is the identity,
which is unbiased with zero variance, so both theorems cover the chain.

Thm. 1: E[FQT gradient | batch] = QAT gradient.
Thm. 2 with the batch fixed (no sampling term):
    Var[grad_W_k] = sum_{l >= k} E[ Var[ Q(dZ_l) gamma^(k,l) | dZ_l ] ],
gamma^(k,l) being the exact backward from dZ_l to grad_W_k (through Q_b1 for
k = l, Q_b2 for k < l).  Given dZ_l that conditional variance is a sum over
code elements of Var[code] (App. C, stochastic rounding) times the squared
norm of the code's response under the linear map: its dequantized
perturbation (S^-1 column, App. B Prop. var) pushed through gamma.
"""
import numpy as np

from . import backward as BW
from . import quantizers as Q
from . import sr
from . import theory


def dequantized_operands(A, W, f_bits=8, theta_bits=8):
    """Xt = Q_f(A), Wt = Q_theta(W) as the float64 values the codes represent."""
    Xt = Q.dequantize(Q.quantize_ptq(np.asarray(A, np.float32), f_bits, False))
    Wt = Q.dequantize(Q.quantize_ptq(np.asarray(W, np.float32), theta_bits, False))
    return Xt, Wt


def layer_forward(A, W, relu, f_bits=8, theta_bits=8):
    """One layer: (Z, Y) in float64, Y = ReLU(Z) when relu else Z."""
    Xt, Wt = dequantized_operands(A, W, f_bits, theta_bits)
    Z = Xt @ Wt.T
    return Z, (np.maximum(Z, 0.0) if relu else Z)


def forward(X, Ws, f_bits=8, theta_bits=8):
    """The chain's layer inputs A_0 .. A_{L-1} (float32, each the rounding of
    the float64 layer output) and the float64 top output Z_{L-1}."""
    acts = [np.asarray(X, np.float32)]
    Z = None
    for i, W in enumerate(Ws):
        last = i == len(Ws) - 1
        Z, Y = layer_forward(acts[-1], W, not last, f_bits, theta_bits)
        if not last:
            acts.append(Y.astype(np.float32))
    return acts, Z


def relu_mask(A):
    return (np.asarray(A) > 0).astype(np.float64)


def qat_backward(acts, Ws, G, f_bits=8, theta_bits=8):
    """QAT gradients (float64) from the layer inputs; returns (grads_W, dZ) per layer."""
    L = len(Ws)
    grads, dZs = [None] * L, [None] * L
    dZ = np.asarray(G, np.float64)
    for i in range(L - 1, -1, -1):
        Xt, Wt = dequantized_operands(acts[i], Ws[i], f_bits, theta_bits)
        dZs[i] = dZ
        grads[i] = dZ.T @ Xt
        if i > 0:
            dZ = (dZ @ Wt) * relu_mask(acts[i])
    return grads, dZs


def fqt_backward(acts, Ws, G, specs, seeds, qb_w=("ptq", 8, 0), f_bits=8, theta_bits=8):
    """FQT gradients: each layer's oracle backward (float64 products of the
    dequantized operands), the next layer down taking the float32 rounding of
    grad_X times the ReLU mask.  Returns (grads_W float64, dZ float32) per layer."""
    L = len(Ws)
    grads, dZs = [None] * L, [None] * L
    dZ = np.asarray(G, np.float32)
    for i in range(L - 1, -1, -1):
        dZs[i] = dZ
        r = BW.linear_backward(acts[i], Ws[i], dZ, specs[i], qb_w, f_bits, theta_bits, seeds[i])
        grads[i] = r["grad_W64"]
        if i > 0:
            dZ = (r["grad_X"] * (np.asarray(acts[i]) > 0)).astype(np.float32)
    return grads, dZs


def response_maps(acts, Ws, l, f_bits=8, theta_bits=8):
    """The exact linear maps gamma^(k,l) for k < l as arrays J_k [N, d_out(l), |W_k|]:
    J_k[n, o] is vec(grad_W_k) when dZ_l is the unit matrix at (n, o).  A
    perturbation of sample n stays in row n through the backward (masks and
    products act per sample), and reaches grad_W_k as an outer product with
    that sample's Xt_k row."""
    ops = [dequantized_operands(acts[i], Ws[i], f_bits, theta_bits) for i in range(l + 1)]
    N = np.asarray(acts[0]).shape[0]
    d_top = Ws[l].shape[0]
    maps = {}
    for k in range(l):
        maps[k] = np.zeros((N, d_top, Ws[k].size))
    masks = [relu_mask(acts[k + 1]) for k in range(l)]
    for n in range(N):
        U = ops[l][1].copy()                                 # row o: dA_l[n] for the unit at (n, o)
        for k in range(l - 1, -1, -1):
            U = U * masks[k][n][None, :]                     # dZ_k[n] per unit
            maps[k][n] = np.einsum("or,c->orc", U, ops[k][0][n]).reshape(d_top, -1)
            U = U @ ops[k][1]                                # dA_k[n] per unit
    return maps


def conditional_variance(J, G, q):
    """Var[ vec(Q(G)) J | G ] exactly: sum over code elements of Var[code] times
    the squared norm of the code's response (its S^-1 column through J)."""
    y = theory.transformed_values(G, q)
    v = sr.exact_var_code(y)
    nrm = (J ** 2).sum(axis=2)                               # [N, d] response norms of unit perturbations
    if q["kind"] == "ptq":
        return float((v * nrm).sum() / float(q["scale"]) ** 2)
    if q["kind"] in ("psq", "shift"):
        return float(((v / q["scale"][:, None].astype(np.float64) ** 2) * nrm).sum())
    total = 0.0
    for info, Si in theory.inverse_scale_blocks(q):
        base, kg, mem = info["base"], info["size"], info["members"]
        R = np.einsum("mq,mod->qod", Si, J[mem])             # response of slot q at column o
        total += float((v[base: base + kg] * (R ** 2).sum(axis=2)).sum())
    return total


def own_layer_variance(A, dZ, qb_w, f_bits=8):
    """Var[grad_W_l | dZ_l] from Q_b1 (per-tensor, element noise independent):
    sum_{n,o} Var[Q_b1(dZ)_no] |Xt_l[n]|^2."""
    Xt = Q.dequantize(Q.quantize_ptq(np.asarray(A, np.float32), f_bits, False))
    q1 = BW.quantize_gradient(np.asarray(dZ, np.float32), qb_w, 0, 0)
    var = theory.exact_elementwise_variance(dZ, q1)
    return float((var * (Xt ** 2).sum(axis=1)[:, None]).sum())


def lower_layer_variances(acts, Ws, l, dZ, spec, f_bits=8, theta_bits=8, maps=None):
    """{k: Var[grad_W_k | dZ_l] from Q_b2(dZ_l) alone} for k < l."""
    if maps is None:
        maps = response_maps(acts, Ws, l, f_bits, theta_bits)
    q2 = BW.quantize_gradient(np.asarray(dZ, np.float32), spec, 0, 1)
    return {k: conditional_variance(J, dZ, q2) for k, J in maps.items()}
