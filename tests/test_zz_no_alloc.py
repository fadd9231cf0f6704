"""The no-allocation entry point fqt_quantize_psq_noalloc against
fqt_quantize_psq (and the oracle), bit for bit, on two calls in a row with
the second input smaller than the first; sizes beyond its fixed scratch are
refused; a non-finite input is reported through its status words."""
import numpy as np
import pytest

from oracle import quantizers as Q

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def fqt():
    from paper_2010_14298_amd import fqt as f
    f.load()
    return f


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def heavy(seed, n, d):
    rng = np.random.default_rng(seed)
    return (rng.lognormal(0, 2, (n, 1)) * rng.standard_normal((n, d))).astype(np.float32)


def test_noalloc_matches_the_workspace_entry_point_on_two_calls():
    f = fqt()
    for rows, cols, bits, seed in ((3000, 1000, 5, 5), (700, 130, 8, 6)):
        x = heavy(seed, rows, cols)
        a = f.fqt_quantize_psq(dev(x), bits, seed=seed, stream=1, code_sum=True)
        b = f.fqt_quantize_psq_noalloc(dev(x), bits, seed=seed, stream=1, code_sum=True)
        for key in ("q", "scale", "zero", "code_sum"):
            np.testing.assert_array_equal(host(b[key]), host(a[key]), err_msg=key)
        assert (host(b["status"]) == 0).all()
        ref = Q.quantize_psq(x, bits, seed=seed, stream=1)
        np.testing.assert_array_equal(host(b["q"]), (ref["code"] - Q.offset(bits)).astype(np.int8))


def test_noalloc_refuses_sizes_beyond_its_scratch_and_reports_bad_data():
    f = fqt()
    big = torch.zeros((300000, 8), dtype=torch.float32, device="cuda")
    with pytest.raises(f.FqtError) as e:
        f.fqt_quantize_psq_noalloc(big, 5)
    assert e.value.code == 2
    x = heavy(7, 40, 16)
    x[3, 5] = np.nan
    b = f.fqt_quantize_psq_noalloc(dev(x), 5)
    assert (host(b["status"]) & 1).any()
    # and a clean call afterwards reports clean data again
    b = f.fqt_quantize_psq_noalloc(dev(heavy(8, 40, 16)), 5)
    assert (host(b["status"]) == 0).all()
