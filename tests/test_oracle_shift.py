"""Pins of the per-tensor-range / per-sample-shift quantizer (Sec. 4.3).

* It is PSQ, code for code, when every row's range is the tensor's range
  over a power of two no larger than 2^E (then s 2^e_i = B / R_i exactly).
* The shifts against an exhaustive search with exact rationals.
* Unbiased (exact mean), and its variance bound between PSQ's and PTQ's.
* Shifted offset codes fit int8, and the contraction identity the grad_W
  epilogue uses: common step 1 / (s 2^E) on the shifted codes plus one
  per-column vector for the per-sample zero points.
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import backward as BW
from oracle import quantizers as Q
from oracle import theory


@pytest.mark.parametrize("bits,E", [(1, 4), (2, 4), (4, 4), (5, 3), (6, 2), (7, 1), (8, 0)])
def test_shift_limit(bits, E):
    assert Q.shift_limit(bits) == E
    half = 1 << (bits - 1)
    assert -half << E >= -128 and (half - 1) << E <= 127


@pytest.mark.parametrize("bits", [4, 5, 6])
def test_equals_psq_when_ranges_are_powers_of_two(bits):
    rng = np.random.default_rng(bits)
    E = Q.shift_limit(bits)
    rows, cols = 24, 40
    m = rng.integers(10 - E, 11, size=rows)
    m[0] = 10                                      # the tensor range: 2^10
    x = np.zeros((rows, cols), np.float32)
    for i in range(rows):
        v = rng.integers(0, 2 ** m[i] + 1, size=cols).astype(np.float64)
        v[0], v[1] = 0, 2 ** m[i]
        x[i] = (v + rng.integers(-500, 500)).astype(np.float32)
    q = Q.quantize_shift(x, bits, seed=7, stream=0)
    p = Q.quantize_psq(x, bits, seed=7, stream=0)
    np.testing.assert_array_equal(q["scale"], p["scale"])
    np.testing.assert_array_equal(q["code"], p["code"])
    np.testing.assert_array_equal(q["shift"], E - (10 - m))


def test_shifts_against_exact_search():
    rng = np.random.default_rng(0)
    for bits in (3, 4, 5):
        E = Q.shift_limit(bits)
        x = (rng.standard_normal((40, 9)) * np.exp(rng.uniform(-4, 2, size=(40, 1)))).astype(np.float32)
        x[5] = 1.5                                 # a constant row: R_i = 0, full shift
        q = Q.quantize_shift(x, bits)
        _, _, R, _ = Q.row_stats(x)
        Rt = Fraction(float(R.max()))
        for i in range(x.shape[0]):
            ok = [e for e in range(E + 1) if Fraction(float(R[i])) * 2 ** e <= Rt]
            assert q["shift"][i] == E - max(ok)
            assert q["scale"][i] == np.float32(float(Q.scale_from_range(R.max(), Q.n_bins(bits))) * 2.0 ** max(ok))


def test_unbiased_and_variance_between_psq_and_ptq():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal((64, 48)) * np.exp(rng.uniform(-3, 1, size=(64, 1)))).astype(np.float32)
    q = Q.quantize_shift(x, 4)
    mean = theory.exact_mean(x, q)
    step = 1.0 / q["scale"][:, None].astype(np.float64)
    # exact up to the float32 rounding of y = s (x - z) (a few ulps of y <= B, in steps)
    assert np.all(np.abs(mean - x) <= step * 2.0 ** -18 + 1e-6 * np.abs(x))
    # a rounding rule off by a fraction of a step would show
    assert np.abs(mean - x).max() < 1e-3 * step.min()
    D = x.shape[1]
    b_psq = theory.matrix_var_bound(Q.quantize_psq(x, 4), D)
    b_shift = theory.matrix_var_bound(q, D)
    b_ptq = theory.matrix_var_bound(dict(Q.quantize_ptq(x, 4, True), code=np.zeros_like(x)), D)
    assert b_psq <= b_shift <= b_ptq
    assert theory.exact_quantizer_variance(x, q) <= b_shift


def test_shifted_contraction_identity():
    rng = np.random.default_rng(2)
    N, d_out, d_in, bits = 50, 12, 9, 4
    G = (rng.standard_normal((N, d_out)) * np.exp(rng.uniform(-3, 1, size=(N, 1)))).astype(np.float32)
    X = rng.standard_normal((N, d_in)).astype(np.float32)
    q = BW.quantize_gradient(G, ("shift", bits, 0), 3, 0)
    qx = Q.quantize_ptq(X, 8, False)
    qs = Q.shifted_codes(q)
    assert qs.min() >= -128 and qs.max() <= 127
    Xr = Q.dequantize(qx)
    ref = Q.dequantize(q).T @ Xr
    E = Q.shift_limit(bits)
    d = 1.0 / (float(q["step_scale"]) * 2.0 ** E)
    zeta = Q.offset(bits) / q["scale"].astype(np.float64) + q["zero"].astype(np.float64)
    got = d * (qs.T @ Xr) + (zeta @ Xr)[None, :]
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())
    r = BW.linear_backward(X, rng.standard_normal((d_out, d_in)).astype(np.float32), G, ("psq", 8, 0),
                           ("shift", bits, 0), seed=3)
    np.testing.assert_array_equal(r["acc_w"], qs.T @ Q.offset_codes(qx))
