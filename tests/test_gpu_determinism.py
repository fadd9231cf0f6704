"""Run-to-run determinism of the whole entry points: the same inputs and seed
give bitwise-identical outputs (no floating-point atomics anywhere; integer
code sums are order-free), and another seed changes them."""
import numpy as np
import pytest

from paper_2010_14298_amd import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def fqt():
    from paper_2010_14298_amd import fqt as f
    f.load()
    return f


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


@pytest.mark.parametrize("qb_x,qb_w", [(("bhq", 5, 64), ("ptq", 8, 0)), (("psq", 4, 0), ("shift", 4, 0)),
                                       (("bhq", 5, 0), ("ptq", 8, 0))])
def test_linear_backward_bitwise_repeatable(qb_x, qb_w):
    f = fqt()
    X, W, G = synth.linear_outlier(seed=3, n=2048, d_in=256, d_out=512)
    dX, dW, dG = dev(X), dev(W), dev(G)
    runs = [f.fqt_linear_backward(dX, dW, dG, qb_x=qb_x, qb_w=qb_w, seed=s)[:2] for s in (5, 5, 6)]
    assert torch.equal(runs[0][0], runs[1][0]) and torch.equal(runs[0][1], runs[1][1])
    assert not torch.equal(runs[0][1], runs[2][1])


def test_conv_backward_bitwise_repeatable():
    f = fqt()
    X, W, G = synth.conv_layer(seed=2, n=16, c=32, h=20, w=20, o=32, k=3, stride=1, pad=1)
    dX, dW, dG = dev(X), dev(W), dev(G)
    runs = [f.fqt_conv_backward_im2col(dX, dW, dG, 1, 1, qb_x=("bhq", 5, 8), seed=s)[:2] for s in (1, 1, 2)]
    assert torch.equal(runs[0][0], runs[1][0]) and torch.equal(runs[0][1], runs[1][1])
    assert not torch.equal(runs[0][1], runs[2][1])


def test_forward_and_chain_bitwise_repeatable():
    f = fqt()
    X, Ws, G = synth.mlp(seed=4, n=512, widths=(96, 128, 64))
    dWs = [dev(W) for W in Ws]
    outs = []
    for _ in range(2):
        acts, Z = f.mlp_forward(dev(X), dWs)
        grads, _ = f.mlp_backward(acts, dWs, dev(G), [("bhq", 4, 8), ("psq", 5, 0)], [7, 8])
        outs.append([Z] + grads)
    for a, b in zip(*outs):
        assert torch.equal(a, b)
