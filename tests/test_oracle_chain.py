"""Pins of the multi-layer chain oracle (CPU).

* The QAT backward against torch autograd of the same network built with the
  straight-through estimator (an independent differentiation).
* The response maps gamma^(k,l) against the QAT backward started at layer l.
* The exact conditional variance through a linear map against Monte Carlo over
  the oracle's own quantizer (PTQ, PSQ, BHQ).
* Thm. 1 and Thm. 2 on the oracle's FQT chain by Monte Carlo over seeds.
"""
import numpy as np
import pytest

from oracle import backward as BW
from oracle import chain as CH
from oracle import quantizers as Q
from paper_2010_14298_amd import synth

torch = pytest.importorskip("torch")

WIDTHS = (6, 10, 8, 5)


def small_chain(seed=0, n=12):
    X, Ws, G = synth.mlp(seed=seed, n=n, widths=WIDTHS)
    acts, _ = CH.forward(X, Ws)
    return X, Ws, G, acts


def test_qat_backward_matches_autograd_with_straight_through():
    X, Ws, G, acts = small_chain()
    t = lambda a: torch.tensor(np.asarray(a, np.float64))
    A = t(acts[0])
    params = []
    Z = None
    for i, W in enumerate(Ws):
        Xt, Wt = CH.dequantized_operands(acts[i], W)
        a_in = A if i == 0 else A_next
        # straight-through: forward value Xt, gradient of the identity
        x_q = a_in + (t(Xt) - a_in).detach()
        w = t(W).requires_grad_(True)
        w_q = w + (t(Wt) - w).detach()
        params.append(w)
        Z = x_q @ w_q.T
        if i < len(Ws) - 1:
            A_next = torch.relu(Z)
            # the chain feeds the float32 rounding of the activation forward; its
            # gradient is the identity
            A_next = A_next + (t(acts[i + 1]) - A_next).detach()
    (Z * t(G)).sum().backward()
    grads, _ = CH.qat_backward(acts, Ws, G)
    for i in range(len(Ws)):
        np.testing.assert_allclose(grads[i], params[i].grad.numpy(), rtol=1e-12, atol=1e-12)


def test_response_maps_reproduce_the_backward_from_layer_l():
    X, Ws, G, acts = small_chain(seed=1)
    rng = np.random.default_rng(3)
    for l in (1, 2):
        maps = CH.response_maps(acts, Ws, l)
        dZ = rng.standard_normal((acts[0].shape[0], Ws[l].shape[0]))
        ref, _ = CH.qat_backward(acts[: l + 1], Ws[: l + 1], dZ)
        for k, J in maps.items():
            got = np.einsum("no,nod->d", dZ, J).reshape(Ws[k].shape)
            np.testing.assert_allclose(got, ref[k], rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("spec", [("ptq", 4, 0), ("psq", 4, 0), ("bhq", 4, 4)])
def test_conditional_variance_matches_monte_carlo(spec):
    X, Ws, G, acts = small_chain(seed=2, n=16)
    l = 2
    dZ = np.asarray(G, np.float32)
    maps = CH.response_maps(acts, Ws, l)
    exact = CH.lower_layer_variances(acts, Ws, l, dZ, spec, maps=maps)
    samples = {k: [] for k in maps}
    for s in range(600):
        g = Q.dequantize(BW.quantize_gradient(dZ, spec, s, 1))
        for k, J in maps.items():
            samples[k].append(np.einsum("no,nod->d", g, J))
    for k in maps:
        emp = float(np.asarray(samples[k]).var(axis=0, ddof=1).sum())
        assert abs(emp - exact[k]) <= 0.12 * exact[k], (k, emp, exact[k])


def test_own_layer_variance_matches_monte_carlo():
    X, Ws, G, acts = small_chain(seed=4, n=16)
    dZ = np.asarray(G, np.float32)
    Xt, _ = CH.dequantized_operands(acts[2], Ws[2])
    exact = CH.own_layer_variance(acts[2], dZ, ("ptq", 4, 0))
    draws = [Q.dequantize(BW.quantize_gradient(dZ, ("ptq", 4, 0), s, 0)).T @ Xt for s in range(600)]
    emp = float(np.asarray(draws).var(axis=0, ddof=1).sum())
    assert abs(emp - exact) <= 0.12 * exact


def test_theorems_on_the_oracle_chain():
    """Thm. 1 (mean over seeds -> QAT gradient) and Thm. 2 (total variance per
    layer = sum of the per-quantizer terms) with the oracle's FQT chain."""
    X, Ws, G, acts = small_chain(seed=5, n=16)
    L = len(Ws)
    specs = [("psq", 4, 0), ("bhq", 4, 4), ("ptq", 5, 0)]
    qb_w = ("ptq", 6, 0)
    S = 400
    qat, _ = CH.qat_backward(acts, Ws, G)
    runs = [CH.fqt_backward(acts, Ws, G, specs, [3 * s + i for i in range(L)], qb_w) for s in range(S)]
    for k in range(L):
        g = np.asarray([r[0][k] for r in runs])
        mean, var = g.mean(axis=0), g.var(axis=0, ddof=1)
        # Thm. 1: |mean - QAT|^2 has expectation sum(var) / S
        assert ((mean - qat[k]) ** 2).sum() <= 3.0 * var.sum() / S
        # Thm. 2: decomposition over the quantizers of layers l >= k
        pred = 0.0
        for l in range(k, L):
            dZs = [r[1][l] for r in runs[:100]] if l < L - 1 else [runs[0][1][l]]
            if l == k:
                pred += np.mean([CH.own_layer_variance(acts[l], d, qb_w) for d in dZs])
            else:
                maps = CH.response_maps(acts, Ws, l)
                pred += np.mean([CH.lower_layer_variances(acts, Ws, l, d, specs[l], maps=maps)[k] for d in dZs])
        assert abs(var.sum() - pred) <= 0.15 * pred, (k, var.sum(), pred)


def test_conditional_variance_keeps_within_group_correlation():
    """BHQ noise is independent per code, not per element: on rows of equal
    scale with one response shared by every sample, the member responses of a
    code add coherently (an element-independent sum is about 12 % off here)."""
    rng = np.random.default_rng(1)
    dZ = rng.standard_normal((16, 5)).astype(np.float32)
    J = np.broadcast_to(np.random.default_rng(0).standard_normal((5, 7)), (16, 5, 7)).copy()
    q = BW.quantize_gradient(dZ, ("bhq", 4, 4), 0, 1)
    exact = CH.conditional_variance(J, dZ, q)
    draws = [np.einsum("no,nod->d", Q.dequantize(BW.quantize_gradient(dZ, ("bhq", 4, 4), s, 1)), J)
             for s in range(3000)]
    emp = float(np.asarray(draws).var(axis=0, ddof=1).sum())
    assert abs(emp - exact) <= 0.05 * exact, (emp, exact)
