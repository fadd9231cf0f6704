"""GPU parity of the quantizers against the oracle (bit-exact codes, scales,
zero points, permutations and code sums), through the C ABI."""
import numpy as np
import pytest

from oracle import quantizers as Q
from paper_2010_14298_amd import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def fqt():
    from paper_2010_14298_amd import fqt as f
    f.load()
    return f


def heavy(seed, n, d):
    rng = np.random.default_rng(seed)
    return (rng.lognormal(0, 2, (n, 1)) * rng.standard_normal((n, d))).astype(np.float32)


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def offset(q):
    return (q["code"] - Q.offset(q["bits"])).astype(np.int8)


SHAPES = [(1, 1), (3, 5), (64, 256), (65, 257), (128, 256), (130, 100), (257, 1030)]


@pytest.mark.parametrize("rows,cols", SHAPES)
@pytest.mark.parametrize("bits", [1, 4, 8])
@pytest.mark.parametrize("stochastic", [0, 1])
def test_ptq(rows, cols, bits, stochastic):
    f = fqt()
    x = heavy(rows * 7 + cols, rows, cols)
    ref = Q.quantize_ptq(x, bits, bool(stochastic), seed=5, stream=3)
    for transpose in (False, True):
        out = f.fqt_quantize_ptq(dev(x), bits, stochastic, seed=5, stream=3, transpose=transpose, code_sum=True)
        q = host(out["q"])
        exp = offset(ref)
        np.testing.assert_array_equal(q, exp.T if transpose else exp)
        assert host(out["scale"])[0] == ref["scale"] and host(out["zero"])[0] == ref["zero"]
        np.testing.assert_array_equal(host(out["code_sum"]), exp.astype(np.int64).sum(axis=0 if transpose else 1))


@pytest.mark.parametrize("rows,cols", SHAPES)
@pytest.mark.parametrize("bits", [2, 4, 5, 8])
def test_psq(rows, cols, bits):
    f = fqt()
    x = heavy(rows + 3 * cols, rows, cols)
    ref = Q.quantize_psq(x, bits, seed=11, stream=1)
    out = f.fqt_quantize_psq(dev(x), bits, seed=11, stream=1, code_sum=True)
    np.testing.assert_array_equal(host(out["q"]), offset(ref))
    np.testing.assert_array_equal(host(out["scale"]), ref["scale"])
    np.testing.assert_array_equal(host(out["zero"]), ref["zero"])
    np.testing.assert_array_equal(host(out["code_sum"]), offset(ref).astype(np.int64).sum(axis=1))


@pytest.mark.parametrize("k", [1, 2, 4, 8, 16, 32, 64])
@pytest.mark.parametrize("rows,cols", [(1, 7), (10, 12), (64, 256), (130, 260), (200, 33), (1000, 64)])
@pytest.mark.parametrize("bits", [4, 5, 8])
def test_bhq(k, rows, cols, bits):
    f = fqt()
    x = heavy(rows * 13 + cols + k, rows, cols)
    ref = Q.quantize_bhq(x, bits, k, seed=3, stream=1)
    out = f.fqt_quantize_bhq(dev(x), bits, k, seed=3, stream=1, code_sum=True)
    np.testing.assert_array_equal(host(out["perm"]), ref["perm"])
    np.testing.assert_array_equal(host(out["group_off"])[: len(ref["group_off"])], ref["group_off"])
    np.testing.assert_array_equal(host(out["scale"]), ref["scale"])
    np.testing.assert_array_equal(host(out["zero"]), ref["zero"])
    np.testing.assert_array_equal(host(out["q"]), offset(ref))
    np.testing.assert_array_equal(host(out["code_sum"]), offset(ref).astype(np.int64).sum(axis=1))


def test_bhq_degenerate_rows():
    # all-zero rows, constant rows, ties in the row norm
    f = fqt()
    x = np.zeros((40, 24), np.float32)
    x[3] = 5.0
    x[7] = np.arange(24)
    x[8] = -np.arange(24)
    x[20:30] = 1e-3 * np.arange(24)
    for k in (4, 16, 64):
        ref = Q.quantize_bhq(x, 5, k, seed=1, stream=1)
        out = f.fqt_quantize_bhq(dev(x), 5, k, seed=1, stream=1)
        np.testing.assert_array_equal(host(out["perm"]), ref["perm"])
        np.testing.assert_array_equal(host(out["scale"]), ref["scale"])
        np.testing.assert_array_equal(host(out["zero"]), ref["zero"])
        np.testing.assert_array_equal(host(out["q"]), offset(ref))


def test_bhq_single_outlier_cube_roots():
    # one dominant row per group exercises lambda1 >> lambda2 and the cube roots
    f = fqt()
    X, W, G = synth.linear_single_outlier(seed=4, n=512, d_in=8, d_out=384)
    for bits in (4, 5, 6, 8):
        ref = Q.quantize_bhq(G, bits, 64, seed=9, stream=1)
        out = f.fqt_quantize_bhq(dev(G), bits, 64, seed=9, stream=1)
        np.testing.assert_array_equal(host(out["scale"]), ref["scale"])
        np.testing.assert_array_equal(host(out["zero"]), ref["zero"])
        np.testing.assert_array_equal(host(out["q"]), offset(ref))


def test_nonfinite_is_reported():
    f = fqt()
    x = heavy(0, 16, 16)
    x[3, 4] = np.nan
    out = f.fqt_quantize_psq(dev(x), 8)
    assert f.fqt_workspace_status(out["ws"]) == 3
    out = f.fqt_quantize_psq(dev(heavy(1, 16, 16)), 8)
    assert f.fqt_workspace_status(out["ws"]) == 0


def test_determinism():
    f = fqt()
    x = dev(heavy(2, 300, 500))
    a = f.fqt_quantize_bhq(x, 5, 64, seed=7, stream=1)
    b = f.fqt_quantize_bhq(x, 5, 64, seed=7, stream=1)
    assert torch.equal(a["q"], b["q"]) and torch.equal(a["perm"], b["perm"])
    c = f.fqt_quantize_bhq(x, 5, 64, seed=8, stream=1)
    assert not torch.equal(a["q"], c["q"])
