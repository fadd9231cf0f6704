"""Exact contraction of 4-bit codes on the 6-bit float matrix cores
(fqt_gemm_s4s4_bf6): accumulators bit-exact to int64 matmul on ragged shapes,
K padding, a K beyond one float32-exact chunk, the extreme codes, and the
data error for a code outside [-8, 7]."""
import numpy as np
import pytest

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


@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (37, 53, 100), (300, 257, 1000), (256, 512, 4096), (129, 65, 128),
                                   (5, 3, 300000)])
def test_bf6_accumulators_exact(M, N, K):
    f = fqt()
    rng = np.random.default_rng(M * 7 + N + K)
    A = rng.integers(-8, 8, size=(M, K), dtype=np.int8)
    B = rng.integers(-8, 8, size=(N, K), dtype=np.int8)
    C, ws = f.fqt_gemm_s4s4_bf6(dev(A), dev(B))
    assert f.fqt_workspace_status(ws) == 0
    np.testing.assert_array_equal(host(C), A.astype(np.int64) @ B.astype(np.int64).T)


def test_bf6_extreme_codes_and_strided_rows():
    f = fqt()
    K = 131072 + 384                              # two float32-exact chunks, products at the maximum
    A = np.full((64, K), -8, np.int8)
    B = np.full((32, K), -8, np.int8)
    B[1] = 7
    C, ws = f.fqt_gemm_s4s4_bf6(dev(A), dev(B))
    assert f.fqt_workspace_status(ws) == 0
    np.testing.assert_array_equal(host(C), A.astype(np.int64) @ B.astype(np.int64).T)
    # row strides larger than K (views into wider buffers)
    rng = np.random.default_rng(3)
    Aw = rng.integers(-8, 8, size=(40, 200), dtype=np.int8)
    Bw = rng.integers(-8, 8, size=(24, 200), dtype=np.int8)
    C2, _ = f.fqt_gemm_s4s4_bf6(dev(Aw)[:, :150], dev(Bw)[:, :150])
    np.testing.assert_array_equal(host(C2), Aw[:, :150].astype(np.int64) @ Bw[:, :150].astype(np.int64).T)


def test_bf6_ffn_shape_sampled_rows():
    """8192 x 1024 x 4096 (the grad_X contraction's shape), sampled rows against int64."""
    f = fqt()
    rng = np.random.default_rng(11)
    A = rng.integers(-8, 8, size=(8192, 4096), dtype=np.int8)
    B = rng.integers(-8, 8, size=(1024, 4096), dtype=np.int8)
    C, ws = f.fqt_gemm_s4s4_bf6(dev(A), dev(B))
    assert f.fqt_workspace_status(ws) == 0
    got = host(C)
    rows = rng.choice(8192, 40, replace=False)
    np.testing.assert_array_equal(got[rows], A[rows].astype(np.int64) @ B.astype(np.int64).T)


@pytest.mark.parametrize("bad", [8, -9, 127, -128])
def test_bf6_code_outside_range_is_a_data_error(bad):
    f = fqt()
    A = np.zeros((16, 64), np.int8)
    B = np.ones((8, 64), np.int8)
    A[3, 17] = bad
    _, ws = f.fqt_gemm_s4s4_bf6(dev(A), dev(B))
    assert f.fqt_workspace_status(ws) == 3
