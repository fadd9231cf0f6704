"""Pins for the oracle's layer backward (Sec. 2.2, Eq. linear-sq-backprop).

* integer accumulators against a brute-force triple loop;
* Theorem 1 (unbiased gradient) for one layer: E[grad] equals the QAT
  gradient of Sec. 2.1 computed from the unquantized G;
* Theorem 2 / Prop. var for one layer: exact output variance against its
  Monte Carlo estimate and against Var[Q_b(G)] |W|_2^2 (Prop. cauchy);
* the dequantized products against the zero-point expansion of the integer
  accumulators (the algebra any int8 contraction must use);
* conv: im2col / col2im against torch's CPU convolution and its input
  gradient (library routines).
"""
import math

import numpy as np
import pytest

from oracle import backward as BW
from oracle import quantizers as Q
from oracle import theory


def small_layer(seed, n=24, d_in=20, d_out=12):
    rng = np.random.default_rng(seed)
    X = np.maximum(rng.standard_normal((n, d_in)), 0).astype(np.float32)
    W = (rng.standard_normal((d_out, d_in)) * 0.3).astype(np.float32)
    s = rng.lognormal(0, 2, (n, 1))
    G = (s * rng.standard_normal((n, d_out))).astype(np.float32)
    return X, W, G


def test_integer_accumulators_brute_force():
    X, W, G = small_layer(0, n=9, d_in=5, d_out=4)
    r = BW.linear_backward(X, W, G, qb_x=("bhq", 5, 4))
    a = Q.offset_codes(r["qb1"])
    b = Q.offset_codes(r["qx"])
    for o in range(4):
        for c in range(5):
            assert r["acc_w"][o, c] == sum(int(a[n, o]) * int(b[n, c]) for n in range(9))
    g2 = Q.offset_codes(r["qb2"])
    w = Q.offset_codes(r["qw"])
    for p in range(9):
        for c in range(5):
            assert r["acc_x"][p, c] == sum(int(g2[p, o]) * int(w[o, c]) for o in range(4))


@pytest.mark.parametrize("kind,k", [("ptq", 0), ("psq", 0), ("bhq", 8)])
def test_theorem1_unbiased_gradients(kind, k):
    X, W, G = small_layer(1)
    r = BW.linear_backward(X, W, G, qb_x=(kind, 4, k))
    Xr, Wr = Q.dequantize(r["qx"]), Q.dequantize(r["qw"])
    EG2 = theory.exact_mean(G, r["qb2"])
    EG1 = theory.exact_mean(G, r["qb1"])
    qat_x = G.astype(np.float64) @ Wr              # QAT gradient, Sec. 2.1
    qat_w = G.astype(np.float64).T @ Xr
    scale_x = np.abs(G).max(axis=1, keepdims=True) * np.abs(Wr).sum(axis=0)[None, :]
    assert (np.abs(EG2 @ Wr - qat_x) <= 1e-5 * scale_x + 1e-12).all()
    assert np.abs(EG1.T @ Xr - qat_w).max() <= 1e-5 * np.abs(G).max() * np.abs(Xr).sum(axis=0).max()


def test_theorem2_single_layer_variance():
    X, W, G = small_layer(2, n=16, d_in=10, d_out=8)
    spec = ("bhq", 4, 8)
    Wr = Q.dequantize(Q.quantize_ptq(W, 8, False))
    q0 = BW.quantize_gradient(G, spec, 0, 1)
    # exact: grad_X = S^-1 (code + c) Wr; Var[grad_X_ic] = sum_p (S^-1)^2_ip sum_o v_po Wr_oc^2
    v = np.zeros(G.shape)
    y = theory.transformed_values(G, q0)
    from oracle import sr
    vc = sr.exact_var_code(y)
    exact = np.zeros((G.shape[0], Wr.shape[1]))
    for info, Si in theory.inverse_scale_blocks(q0):
        base, kg, mem = info["base"], info["size"], info["members"]
        exact[mem] = (Si ** 2) @ (vc[base: base + kg] @ (Wr ** 2))
    seeds = 600
    vals = np.stack([Q.dequantize(BW.quantize_gradient(G, spec, s, 1)) @ Wr for s in range(seeds)])
    mc = vals.var(axis=0, ddof=1).sum()
    assert abs(mc - exact.sum()) / exact.sum() < 0.1
    # Prop. cauchy: Var[Q(G) W] <= Var[Q(G)] |W|_2^2
    qv = theory.exact_quantizer_variance(G, q0)
    assert exact.sum() <= qv * np.linalg.norm(Wr, 2) ** 2 * (1 + 1e-9)


@pytest.mark.parametrize("kind,k", [("ptq", 0), ("psq", 0), ("bhq", 4), ("bhq", 1)])
def test_zero_point_expansion_matches_dequantized_products(kind, k):
    X, W, G = small_layer(3, n=19, d_in=7, d_out=9)
    r = BW.linear_backward(X, W, G, qb_x=(kind, 5, k))
    qx, qw, qb1, qb2 = r["qx"], r["qw"], r["qb1"], r["qb2"]
    # grad_W: per-tensor times per-tensor, four terms
    dG, dX = 1.0 / float(qb1["scale"]), 1.0 / float(qx["scale"])
    zG = float(qb1["zero"]) + 128 * dG
    zX = float(qx["zero"]) + 128 * dX
    sG = Q.offset_codes(qb1).sum(axis=0)           # per d_out column
    sX = Q.offset_codes(qx).sum(axis=0)            # per d_in column
    N = X.shape[0]
    gw = dG * dX * r["acc_w"] + dG * zX * sG[:, None] + zG * dX * sX[None, :] + N * zG * zX
    np.testing.assert_allclose(gw, r["grad_W64"], rtol=1e-12, atol=1e-12 * np.abs(gw).max())
    # grad_X: per-row (or per-group) quantizer times per-tensor weights
    dW = 1.0 / float(qw["scale"])
    zW = float(qw["zero"]) + 128 * dW
    sW = Q.offset_codes(qw).sum(axis=0)            # per d_in column, over d_out
    d_out = W.shape[0]
    half = 1 << (qb2["bits"] - 1)
    rowsum = Q.offset_codes(qb2).sum(axis=1)
    if kind in ("ptq", "psq"):
        s = np.broadcast_to(np.asarray(qb2["scale"], np.float64), (N,))
        z = np.broadcast_to(np.asarray(qb2["zero"], np.float64), (N,))
        dg = 1.0 / s
        zg = z + half * dg
        gx = (dg * dW)[:, None] * r["acc_x"] + (dg * zW * rowsum)[:, None] + zg[:, None] * (dW * sW + d_out * zW)[None, :]
    else:
        # per slot T = (code + c) W~, then diag(1/d) Q per group, rows back through perm
        gx = np.zeros((N, X.shape[1]))
        for info in qb2["plan"]["groups"]:
            base, kg, mem = info["base"], info["size"], info["members"]
            sl = slice(base, base + kg)
            d = qb2["scale"][sl].astype(np.float64)
            if kg == 1:
                dg = 1.0 / d[0]
                zg = float(qb2["zero"][base]) + half * dg
                gx[mem[0]] = dg * dW * r["acc_x"][base] + dg * zW * rowsum[base] + zg * (dW * sW + d_out * zW)
                continue
            h = half + float(qb2["zero"][base])
            T = dW * r["acc_x"][sl] + zW * rowsum[sl][:, None] + h * (dW * sW + d_out * zW)[None, :]
            a = 1.0 / math.sqrt(kg)
            tau = (a * T.sum(axis=0) - T[0]) / (1.0 - a)
            Z = T - a * tau[None, :]
            Z[0] = T[0] + (1.0 - a) * tau
            gx[mem] = Z / d[:, None]
    np.testing.assert_allclose(gx, r["grad_X64"], rtol=1e-9, atol=1e-10 * np.abs(gx).max())


def test_grad_x_matches_bifurcated_definition_small_config():
    # grad_X uses Q_b2 (stream 1), grad_W uses Q_b1 (stream 0): App. E
    X, W, G = small_layer(4)
    r = BW.linear_backward(X, W, G, qb_x=("psq", 8, 0), seed=5)
    q1 = Q.quantize_ptq(G, 8, True, seed=5, stream=0)
    q2 = Q.quantize_psq(G, 8, seed=5, stream=1)
    np.testing.assert_array_equal(r["qb1"]["code"], q1["code"])
    np.testing.assert_array_equal(r["qb2"]["code"], q2["code"])


# ----------------------------------------------------------------------------
# conv
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("k,stride,pad", [(3, 1, 1), (1, 2, 0), (3, 2, 1), (7, 2, 3)])
def test_im2col_col2im_against_torch(k, stride, pad):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(k + stride)
    n, h, w, c, o = 2, 9, 8, 3, 4
    x = rng.standard_normal((n, h, w, c))
    wt = rng.standard_normal((o, k, k, c))
    ho, wo = BW.conv_out_size(h, k, stride, pad), BW.conv_out_size(w, k, stride, pad)
    cols = BW.im2col(x, k, k, stride, pad, ho, wo)
    y = (cols @ wt.reshape(o, -1).T).reshape(n, ho, wo, o)
    xt = torch.from_numpy(x).permute(0, 3, 1, 2)
    wtt = torch.from_numpy(wt).permute(0, 3, 1, 2)
    yt = torch.nn.functional.conv2d(xt, wtt, stride=stride, padding=pad).permute(0, 2, 3, 1).numpy()
    np.testing.assert_allclose(y, yt, rtol=1e-10, atol=1e-10)
    g = rng.standard_normal((n, ho, wo, o))
    gx = BW.col2im(g.reshape(-1, o) @ wt.reshape(o, -1), n, h, w, c, k, k, stride, pad, ho, wo)
    gt = torch.nn.grad.conv2d_input((n, c, h, w), wtt, torch.from_numpy(g).permute(0, 3, 1, 2),
                                    stride=stride, padding=pad).permute(0, 2, 3, 1).numpy()
    np.testing.assert_allclose(gx, gt, rtol=1e-10, atol=1e-10)
    gw = (g.reshape(-1, o).T @ cols).reshape(o, k, k, c)
    gwt = torch.nn.grad.conv2d_weight(xt, (o, c, k, k), torch.from_numpy(g).permute(0, 3, 1, 2),
                                      stride=stride, padding=pad).permute(0, 2, 3, 1).numpy()
    np.testing.assert_allclose(gw, gwt, rtol=1e-10, atol=1e-10)


def test_conv_backward_unbiased_and_accumulators():
    rng = np.random.default_rng(5)
    n, h, w, c, o = 4, 5, 5, 3, 2
    X = np.maximum(rng.standard_normal((n, h, w, c)), 0).astype(np.float32)
    W = rng.standard_normal((o, 3, 3, c)).astype(np.float32)
    G = (rng.lognormal(0, 2, (n, 1, 1, 1)) * rng.standard_normal((n, h, w, o))).astype(np.float32)
    r = BW.conv_backward(X, W, G, 1, 1, qb_x=("bhq", 5, 2))
    # accumulators: brute force over output pixels and taps (padding contributes 0)
    a = Q.offset_codes(r["qb1"]).reshape(n, h, w, o)
    b = Q.offset_codes(r["qx"]).reshape(n, h, w, c)
    acc = np.zeros((o, 3, 3, c), np.int64)
    for nn in range(n):
        for y in range(h):
            for x in range(w):
                for rr in range(3):
                    for ss in range(3):
                        iy, ix = y - 1 + rr, x - 1 + ss
                        if 0 <= iy < h and 0 <= ix < w:
                            acc[:, rr, ss, :] += np.outer(a[nn, y, x], b[nn, iy, ix])
    np.testing.assert_array_equal(acc, r["acc_w"])
    # Theorem 1 through the conv: E[grad_X] is the QAT input gradient
    EG2 = theory.exact_mean(G.reshape(n, -1), r["qb2"]).reshape(-1, o)
    Wr = Q.dequantize(r["qw"]).reshape(o, -1)
    e = BW.col2im(EG2 @ Wr, n, h, w, c, 3, 3, 1, 1, h, w)
    qat = BW.col2im(G.reshape(-1, o).astype(np.float64) @ Wr, n, h, w, c, 3, 3, 1, 1, h, w)
    assert np.abs(e - qat).max() <= 1e-5 * np.abs(qat).max()


def test_conv_backward_per_sample_grad_w_unbiased():
    # per-sample Q_b1 on the conv (one scale per sample, Sec. 4.1): Theorem 1
    # through grad_W, whose expectation is the QAT weight gradient G^T im2col(X~)
    rng = np.random.default_rng(6)
    n, h, w, c, o = 5, 6, 6, 3, 2
    X = np.maximum(rng.standard_normal((n, h, w, c)), 0).astype(np.float32)
    W = rng.standard_normal((o, 3, 3, c)).astype(np.float32)
    G = (rng.lognormal(0, 2, (n, 1, 1, 1)) * rng.standard_normal((n, 3, 3, o))).astype(np.float32)
    r = BW.conv_backward(X, W, G, 2, 1, qb_x=("ptq", 8, 0), qb_w=("psq", 8, 0))
    assert r["qb1"]["scale"].shape == (n,)
    cols = BW.im2col(Q.dequantize(r["qx"]).reshape(n, h, w, c), 3, 3, 2, 1, 3, 3)
    EG1 = theory.exact_mean(G.reshape(n, -1), r["qb1"]).reshape(-1, o)
    qat = G.reshape(-1, o).astype(np.float64).T @ cols
    assert np.abs(EG1.T @ cols - qat).max() <= 1e-5 * np.abs(qat).max()
    # each sample's rows dequantize on their own grid: step 1 / s_i from its range
    G1r = Q.dequantize(r["qb1"]).reshape(n, -1)
    for i in range(n):
        R = float(G[i].max()) - float(G[i].min())
        assert np.abs(G1r[i] - G[i].reshape(-1)).max() <= R / 255 * (1 + 1e-6)
