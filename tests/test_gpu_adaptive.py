"""GPU parity of the general block Householder plans: App. D's adaptive groups
(every number of groups G scored on the device) and fixed block sizes that
are not a power of two up to 64.  The objective of every G, the chosen G, the
plan (perm, per-slot scale and zero, group offsets) and the codes equal the
oracle's bit for bit; the linear and conv backward with these plans match the
oracle within 1e-5 row-normwise."""
import numpy as np
import pytest

from oracle import backward as BW
from oracle import quantizers as Q
from paper_2010_14298_amd import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
REL_TOL = 1e-5


def fqt():
    from paper_2010_14298_amd import fqt as f
    f.load()
    return f


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def offset(q):
    return (q["code"] - Q.offset(q["bits"])).astype(np.int8)


def rownorm_err(got, ref):
    got = got.reshape(got.shape[0], -1).astype(np.float64)
    ref = ref.reshape(ref.shape[0], -1).astype(np.float64)
    den = np.abs(ref).max(axis=1)
    num = np.abs(got - ref).max(axis=1)
    return float(np.max(np.where(den > 0, num / np.where(den > 0, den, 1), num)))


def matrices():
    rng = np.random.default_rng(11)
    out = {
        "lognormal_rows": (rng.lognormal(0, 2, (300, 1)) * rng.standard_normal((300, 96))).astype(np.float32),
        "gaussian": rng.standard_normal((257, 64)).astype(np.float32),
        "zeros": np.zeros((70, 16), np.float32),
        "one_row": rng.standard_normal((1, 33)).astype(np.float32),
    }
    _, _, out["outliers_1pct"] = synth.linear_outlier(seed=2, n=400, d_in=8, d_out=128)
    _, _, out["single_outlier"] = synth.linear_single_outlier(seed=3, n=256, d_in=8, d_out=256)
    return out


def check_plan(out, ref):
    np.testing.assert_array_equal(host(out["perm"]), ref["perm"])
    np.testing.assert_array_equal(host(out["scale"]), ref["scale"])
    np.testing.assert_array_equal(host(out["zero"]), ref["zero"])
    G = int(host(out["num_groups"])[0])
    assert G == ref["G"]
    np.testing.assert_array_equal(host(out["group_off"])[: G + 1], ref["group_off"])
    np.testing.assert_array_equal(host(out["q"]), offset(ref))


@pytest.mark.parametrize("name", ["lognormal_rows", "gaussian", "zeros", "one_row", "outliers_1pct",
                                  "single_outlier"])
@pytest.mark.parametrize("bits", [4, 5, 8])
def test_appd_objective_choice_plan_and_codes(name, bits):
    f = fqt()
    x = matrices()[name]
    G_ref, obj_ref = Q.bhq_appd(x, bits)
    G, obj, _ = f.fqt_bhq_adaptive_groups(dev(x), bits)
    np.testing.assert_array_equal(host(obj), np.array(obj_ref, np.float64))
    assert int(host(G)[0]) == G_ref
    out = f.fqt_quantize_bhq(dev(x), bits, 0, seed=5, stream=1)
    check_plan(out, Q.quantize_bhq(x, bits, 0, seed=5, stream=1))


@pytest.mark.parametrize("k", [3, 5, 48, 100, 1000])
def test_fixed_block_general_layout(k):
    # block sizes the aligned tiles do not take go through the general plan
    f = fqt()
    x = matrices()["lognormal_rows"]
    for bits in (4, 5, 8):
        out = f.fqt_quantize_bhq(dev(x), bits, k, seed=6, stream=1)
        check_plan(out, Q.quantize_bhq(x, bits, k, seed=6, stream=1))


@pytest.mark.parametrize("k", [0, 64])
def test_twenty_thousand_rows(k):
    # above the one-launch ranking limit (16384 rows): chunk sorts and rank merge;
    # App. D sampled at G values the oracle evaluates one by one
    f = fqt()
    _, _, x = synth.linear_outlier(seed=7, n=20000, d_in=8, d_out=40)
    out = f.fqt_quantize_bhq(dev(x), 5, k, seed=3, stream=1)
    if k == 0:
        G, obj, _ = f.fqt_bhq_adaptive_groups(dev(x), 5)
        obj = host(obj)
        G = int(host(G)[0])
        # the device's choice is the argmin of its own scores, ties to fewer groups
        assert G == int(np.argmin(obj)) + 1
        _, R, M, order = Q._sorted_rows(x)
        P = Q.appd_prefix(M[order])
        for g in sorted({1, 2, 3, 199, 5000, G - 1, G, G + 1, 20000} & set(range(1, 20001))):
            assert obj[g - 1] == Q.appd_objective(R, M, order, P, 5, g), g
        ref = Q.quantize_bhq(x, 5, 0, seed=3, stream=1, plan=Q.bhq_appd_plan(x, 5, G))
    else:
        ref = Q.quantize_bhq(x, 5, k, seed=3, stream=1)
    check_plan(out, ref)


def test_adaptive_nonfinite_is_reported():
    f = fqt()
    x = np.ones((20, 8), np.float32)
    x[4, 2] = np.inf
    _, _, ws = f.fqt_bhq_adaptive_groups(dev(x), 5)
    assert f.fqt_workspace_status(ws) == 3
    # the plan over bad data is still a permutation
    out = f.fqt_quantize_bhq(dev(x), 5, 0)
    assert sorted(host(out["perm"]).tolist()) == list(range(20))
    assert f.fqt_workspace_status(out["ws"]) == 3


@pytest.mark.parametrize("shape", [(128, 256, 256), (300, 64, 128), (1000, 96, 200)])
@pytest.mark.parametrize("block", [0, 48])
def test_linear_backward_general_plan(shape, block):
    N, d_in, d_out = shape
    X, W, G = synth.linear_small(seed=N, n=N, d_in=d_in, d_out=d_out)
    qb_x = ("bhq", 5, block)
    r = BW.linear_backward(X, W, G, qb_x=qb_x, seed=1)
    f = fqt()
    gW, gX, ws = f.fqt_linear_backward(dev(X), dev(W), dev(G), qb_x=qb_x, seed=1)
    assert f.fqt_workspace_status(ws) == 0
    assert rownorm_err(host(gW), r["grad_W64"]) <= REL_TOL
    assert rownorm_err(host(gX), r["grad_X64"]) <= REL_TOL


def test_linear_backward_general_plan_relu_mask():
    X, W, G = synth.linear_small(seed=5, n=200, d_in=64, d_out=96)
    qb_x = ("bhq", 4, 0)
    r = BW.linear_backward(X, W, G, qb_x=qb_x, seed=4)
    f = fqt()
    _, gX, _ = f.fqt_linear_backward(dev(X), dev(W), dev(G), qb_x=qb_x, seed=4, relu_input=True)
    ref = np.where(X > 0, r["grad_X64"], 0.0)
    assert rownorm_err(host(gX), ref) <= REL_TOL
    assert (host(gX)[X <= 0] == 0).all()


@pytest.mark.parametrize("block", [0, 12])
def test_conv_backward_general_plan(block):
    X, W, G = synth.conv_layer(seed=3, n=40, c=16, h=6, w=6, o=16, k=3, stride=1, pad=1)
    qb_x = ("bhq", 5, block)
    r = BW.conv_backward(X, W, G, 1, 1, qb_x=qb_x, seed=2)
    f = fqt()
    gW, gX, ws = f.fqt_conv_backward_im2col(dev(X), dev(W), dev(G), 1, 1, qb_x=qb_x, seed=2)
    assert f.fqt_workspace_status(ws) == 0
    assert rownorm_err(host(gW), r["grad_W64"]) <= REL_TOL
    assert rownorm_err(host(gX), r["grad_X64"]) <= REL_TOL


def test_conv_backward_general_plan_many_samples():
    # 150 samples: more slots per input pixel than one 128-row tile holds,
    # so App. D groups cross tile boundaries of the input-gradient contraction
    X, W, G = synth.conv_layer(seed=4, n=150, c=16, h=5, w=5, o=32, k=3, stride=2, pad=1)
    qb_x = ("bhq", 4, 0)
    r = BW.conv_backward(X, W, G, 2, 1, qb_x=qb_x, seed=8)
    f = fqt()
    gW, gX, ws = f.fqt_conv_backward_im2col(dev(X), dev(W), dev(G), 2, 1, qb_x=qb_x, seed=8)
    assert f.fqt_workspace_status(ws) == 0
    assert rownorm_err(host(gW), r["grad_W64"]) <= REL_TOL
    assert rownorm_err(host(gX), r["grad_X64"]) <= REL_TOL
