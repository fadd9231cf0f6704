"""Pins for the oracle's PTQ / PSQ / BHQ against what the paper fixes.

* unbiasedness E[Q(X)] = X (Sec. 2.2 requires an unbiased Q_b) from the exact
  expectation, and from the mean over many seeds;
* the exact quantizer variance against its Monte Carlo estimate and against
  the bounds of Eq. (variance-scale-shift), Sec. 4.1, Eq.
  (matrix-quantizer-variance) and Sec. 4.2;
* the Householder reflection's identities (Sec. 4.2) on an explicit matrix;
* the closed-form s1, s2 (App. C.4) against the constraint they solve and
  against a brute-force minimisation;
* reductions: PSQ with one row is PTQ; BHQ with block size 1 is PSQ;
* the correctly rounded cube root against 60-digit decimal arithmetic.
"""
import decimal
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import quantizers as Q
from oracle import sr, theory


def heavy_rows(seed, n, d, sigma=2.0):
    rng = np.random.default_rng(seed)
    s = rng.lognormal(0, sigma, size=(n, 1))
    return (s * rng.standard_normal((n, d))).astype(np.float32)


# ----------------------------------------------------------------------------
# PTQ / PSQ
# ----------------------------------------------------------------------------

def test_ptq_deterministic_endpoints():
    x = heavy_rows(0, 7, 13)
    for bits in (1, 4, 8):
        q = Q.quantize_ptq(x, bits, stochastic=False)
        B = Q.n_bins(bits)
        assert q["code"].min() == 0 and q["code"].max() == B
        assert q["code"][np.unravel_index(np.argmin(x), x.shape)] == 0
        assert q["code"][np.unravel_index(np.argmax(x), x.shape)] == B
        # a deterministic quantizer is within half a bin of the input
        err = np.abs(Q.dequantize(q) - x)
        assert err.max() <= 0.5 / float(q["scale"]) * (1 + 1e-5)


def test_ptq_degenerate_constant_tensor():
    x = np.full((3, 4), 2.5, np.float32)
    q = Q.quantize_ptq(x, 8, stochastic=True, seed=1)
    assert float(q["scale"]) == 1.0 and (q["code"] == 0).all()
    np.testing.assert_array_equal(Q.dequantize(q), x)


def test_psq_single_row_is_ptq():
    x = heavy_rows(1, 1, 300)
    for bits in (2, 5, 8):
        a = Q.quantize_psq(x, bits, seed=9, stream=1)
        b = Q.quantize_ptq(x, bits, True, seed=9, stream=1)
        np.testing.assert_array_equal(a["code"], b["code"])
        assert a["scale"][0] == b["scale"] and a["zero"][0] == b["zero"]


@pytest.mark.parametrize("kind", ["ptq", "psq"])
def test_affine_unbiased_exact_mean(kind):
    x = heavy_rows(2, 6, 40)
    q = Q.quantize_ptq(x, 4, True) if kind == "ptq" else Q.quantize_psq(x, 4)
    m = theory.exact_mean(x, q)
    # exact up to the float32 evaluation of s (x - z) and the 2^-24 SR excess
    scale = np.broadcast_to(np.asarray(q["scale"], np.float64).reshape(-1, 1), x.shape)
    zero = np.broadcast_to(np.asarray(q["zero"], np.float64).reshape(-1, 1), x.shape)
    tol = (2.0 ** -22) * (np.abs(x - zero) + 1.0 / scale) + 2.0 ** -24 / scale
    assert (np.abs(m - x) <= tol).all()


def test_ptq_psq_variance_bounds_and_order():
    x = heavy_rows(3, 32, 64)
    for bits in (4, 8):
        qp = Q.quantize_ptq(x, bits, True)
        qs = Q.quantize_psq(x, bits)
        vp = theory.exact_quantizer_variance(x, qp)
        vs = theory.exact_quantizer_variance(x, qs)
        assert vp <= theory.ptq_var_bound(x, bits) * (1 + 1e-9)
        assert vs <= theory.psq_var_bound(x, bits) * (1 + 1e-9)
        assert vs <= theory.matrix_var_bound(qs, x.shape[1]) * (1 + 1e-9)
        assert vs < vp


def test_each_fewer_bit_roughly_quadruples_variance():
    # Sec. 3.3: the bound scales with 1 / B^2
    x = heavy_rows(4, 16, 256)
    v = [theory.exact_quantizer_variance(x, Q.quantize_psq(x, b)) for b in (4, 5, 6, 7, 8)]
    ratios = np.array(v[:-1]) / np.array(v[1:])
    assert ((ratios > 3.0) & (ratios < 5.5)).all()


# ----------------------------------------------------------------------------
# Householder reflection and BHQ scalars
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("k", [2, 3, 8, 64])
def test_householder_identities(k):
    H = theory.householder_matrix(k)
    np.testing.assert_allclose(H, H.T, atol=1e-15)
    np.testing.assert_allclose(H @ H, np.eye(k), atol=1e-14)
    e1 = np.zeros(k)
    e1[0] = 1
    np.testing.assert_allclose(H @ e1, np.full(k, 1 / math.sqrt(k)), atol=1e-15)
    x = np.random.default_rng(k).standard_normal(k)
    assert abs(np.linalg.norm(H @ x) - np.linalg.norm(x)) < 1e-13


@pytest.mark.parametrize("k", [2, 5, 64])
def test_bhq_dequant_applies_the_reflection(k):
    # the rank-1 inverse in dequantize_bhq equals diag(1/d) H (code + c) with
    # the explicit matrix
    x = heavy_rows(5, k, 9)
    q = Q.quantize_bhq(x, 5, k, seed=2)
    info = q["plan"]["groups"][0]
    d = q["scale"][:k].astype(np.float64)
    w = q["code"][:k].astype(np.float64) + float(q["zero"][0])
    ref = np.diag(1 / d) @ theory.householder_matrix(k) @ w
    got = Q.dequantize_bhq(q)[info["members"]]
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


def test_bhq_forward_transform_is_scaled_reflection():
    k = 16
    x = heavy_rows(6, k, 33)
    plan = Q.bhq_plan(x, 5, k)
    info = dict(plan["groups"][0], k=k)
    y = Q.bhq_transform(x[info["members"]], info)
    d = plan["scale"][:k].astype(np.float64)
    ref = theory.householder_matrix(k) @ (d[:, None] * x[info["members"]].astype(np.float64)) - float(info["cg"])
    assert np.abs(y - ref).max() <= 2.0 ** -18 * np.abs(ref).max()


def test_cbrt_correctly_rounded():
    decimal.getcontext().prec = 60
    rng = np.random.default_rng(0)
    xs = np.concatenate([rng.uniform(0, 1, 300), rng.lognormal(0, 20, 300), [1.0, 8.0, 27.0, 1e-30, 3e38]])
    for x in xs.astype(np.float32):
        if x == 0:
            continue
        r = Q.cbrt_rn(x)
        exact = decimal.Decimal(float(x)) ** (decimal.Decimal(1) / 3)
        best = min((np.nextafter(r, np.float32(0)), r, np.nextafter(r, np.float32(np.inf))),
                   key=lambda c: abs(decimal.Decimal(float(c)) - exact))
        assert best == r, (x, r, best)
    assert Q.cbrt_rn(np.float32(27.0)) == np.float32(3.0)
    assert Q.cbrt_rn(np.float32(0.125)) == np.float32(0.5)


def test_householder_scales_solve_the_constraint_and_minimise():
    # App. C.4: lambda1 s1 / sqrt(k) + lambda2 s2 sqrt(k) = B, and the pair
    # minimises s1^-2 + k s2^-2 on that line
    B, k = 31, 64
    x = np.zeros((k, 50), np.float32)
    rng = np.random.default_rng(1)
    x[0] = 100 * rng.standard_normal(50)
    x[1:] = 0.3 * rng.standard_normal((k - 1, 50))
    plan = Q.bhq_plan(x, 5, k)
    g = plan["groups"][0]
    lam1, lam2, s1, s2 = (float(g[t]) for t in ("lam1", "lam2", "s1", "s2"))
    lhs = lam1 * s1 / math.sqrt(k) + lam2 * s2 * math.sqrt(k)
    assert abs(lhs - B) < 1e-5 * B
    f = lambda a: a ** -2 + k * ((B - lam1 * a / math.sqrt(k)) / (lam2 * math.sqrt(k))) ** -2
    grid = np.linspace(0.2 * s1, min(1.8 * s1, 0.999 * B * math.sqrt(k) / lam1), 4001)
    assert f(s1) <= min(f(a) for a in grid) * (1 + 1e-6)


def test_bhq_range_invariant():
    # App. C.4's bound puts every transformed value in [c_g, c_g + B]
    x = heavy_rows(7, 256, 64)
    for bits, k in ((5, 64), (4, 16), (8, 8)):
        q = Q.quantize_bhq(x, bits, k, seed=0)
        y = theory.transformed_values(x, q)
        B = Q.n_bins(bits)
        assert y.min() >= -1e-4 * B and y.max() <= B * (1 + 1e-4)


def test_bhq_block_one_is_psq():
    x = heavy_rows(8, 40, 24)
    a = Q.quantize_bhq(x, 5, 1, seed=4, stream=1)
    b = Q.quantize_psq(x, 5, seed=4, stream=1)
    perm = a["perm"]
    np.testing.assert_array_equal(a["code"], b["code"][perm])
    np.testing.assert_array_equal(a["scale"], b["scale"][perm])
    np.testing.assert_array_equal(a["zero"], b["zero"][perm])
    np.testing.assert_array_equal(Q.dequantize(a), Q.dequantize(b))


def test_bhq_grouping_layout():
    x = heavy_rows(9, 130, 8)
    q = Q.quantize_bhq(x, 5, 64)
    sizes = np.diff(q["group_off"])
    np.testing.assert_array_equal(sizes, [64, 64, 2])
    M = np.abs(x).max(axis=1)
    order = sorted(range(130), key=lambda i: (-M[i], i))
    assert list(q["perm"][[0, 64, 128]]) == order[:3]          # large rows lead their group
    assert sorted(q["perm"]) == list(range(130))
    G, sz = Q.bhq_groups(130, 64)
    assert G == 3 and sz == [64, 64, 2]
    assert Q.bhq_groups(100, 64) == (2, [64, 36])
    assert Q.bhq_groups(10, 4) == (3, [4, 4, 2])
    assert Q.bhq_groups(9, 4) == (3, [4, 4, 1])


def test_bhq_degenerate_groups():
    # zero small rows, constant large row, all-zero group
    x = np.zeros((8, 6), np.float32)
    x[0] = np.arange(6)
    x[4] = 3.0
    q = Q.quantize_bhq(x, 4, 4, seed=1)
    for g in q["plan"]["groups"]:
        assert np.isfinite(g["s1"]) and np.isfinite(g["s2"]) and np.isfinite(g["cg"])
    np.testing.assert_allclose(theory.exact_mean(x, q), x, atol=1e-5)


def test_bhq_unbiased_exact_mean():
    x = heavy_rows(10, 128, 32)
    q = Q.quantize_bhq(x, 5, 64)
    m = theory.exact_mean(x, q)
    # float32 transform rounding only: a few ulps of the group's largest value
    for g in q["plan"]["groups"]:
        mem = g["members"]
        scale = np.abs(x[mem]).max()
        assert np.abs(m[mem] - x[mem]).max() <= 2.0 ** -19 * scale


def test_bhq_variance_bounds_single_outlier():
    # Sec. 4.2: one dominant row; BHQ << PSQ << PTQ and the bound of App. C.4
    rng = np.random.default_rng(11)
    n, d, bits = 64, 128, 5
    x = (0.01 * rng.standard_normal((n, d))).astype(np.float32)
    x[17] = 100 * rng.standard_normal(d)
    qb = Q.quantize_bhq(x, bits, n)
    qs = Q.quantize_psq(x, bits)
    qp = Q.quantize_ptq(x, bits, True)
    vb, vs, vp = (theory.exact_quantizer_variance(x, q) for q in (qb, qs, qp))
    assert vb < vs / 10 and vs < vp / 10
    assert vb <= theory.matrix_var_bound(qb, d) * (1 + 1e-9)
    g = qb["plan"]["groups"][0]
    assert vb <= theory.householder_var_bound(float(g["lam1"]), float(g["lam2"]), n, d, bits) * (1 + 1e-6)
    # order of lambda1^2 D / (4 B^2 N)
    B = Q.n_bins(bits)
    approx = float(g["lam1"]) ** 2 * d / (4 * B * B * n)
    assert vb < 2 * approx


def test_exact_variance_brute_force_tiny():
    # enumerate all 2^(N D) SR outcomes of a 2 x 3 BHQ group (b = 2) and of PSQ
    x = np.float32([[1.5, -2.0, 0.25], [0.1, -0.05, 0.2]])
    for q in (Q.quantize_bhq(x, 2, 2), Q.quantize_psq(x, 2), Q.quantize_ptq(x, 2, True)):
        y = theory.transformed_values(x, q)
        p = sr.round_up_probability(y).ravel()
        fl = np.floor(y).astype(np.float64).ravel()
        B = Q.n_bins(q["bits"])
        mean = np.zeros(x.shape)
        second = np.zeros(x.shape)
        for bits in itertools.product([0, 1], repeat=x.size):
            b = np.array(bits, np.float64)
            prob = float(np.prod(np.where(b == 1, p, 1 - p)))
            code = np.clip(fl + b, 0, B).reshape(x.shape)
            val = Q.dequantize(dict(q, code=code))
            mean += prob * val
            second += prob * val ** 2
        np.testing.assert_allclose(mean, theory.exact_mean(x, q), atol=1e-12)
        np.testing.assert_allclose((second - mean ** 2).sum(), theory.exact_quantizer_variance(x, q), rtol=1e-9)
        np.testing.assert_allclose(mean, x, atol=1e-5)


@pytest.mark.parametrize("kind", ["ptq", "psq", "bhq"])
def test_monte_carlo_mean_and_variance(kind):
    x = heavy_rows(12, 16, 24)
    seeds = 400
    f = {"ptq": lambda s: Q.quantize_ptq(x, 4, True, seed=s),
         "psq": lambda s: Q.quantize_psq(x, 4, seed=s),
         "bhq": lambda s: Q.quantize_bhq(x, 4, 8, seed=s)}[kind]
    vals = np.stack([Q.dequantize(f(s)) for s in range(seeds)])
    q0 = f(0)
    ev = theory.exact_mean(x, q0)
    var_el = vals.var(axis=0, ddof=1)
    exact_el = theory.exact_elementwise_variance(x, q0)
    # mean: z-test per element against the exact mean with the exact variance
    se = np.sqrt(exact_el / seeds)
    live = se > 1e-12 * np.abs(x).max()
    z = np.abs(vals.mean(axis=0) - ev)[live] / se[live]
    assert (z < 5.5).all()
    # elements with no variance never move
    assert np.abs(vals.std(axis=0)[~live]).max(initial=0) < 1e-9 * np.abs(x).max()
    np.testing.assert_allclose(ev, x, rtol=0, atol=1e-4 * np.abs(x).max())
    # total variance within a few percent of the closed form
    tv = exact_el.sum()
    assert abs(var_el.sum() - tv) / tv < 0.1


# ---------------------------------------------------------------------------
# group column sum: one slot at a time, in slot order
# ---------------------------------------------------------------------------
def test_group_column_sum_is_sequential_in_slot_order():
    # float32 values whose sum depends on the order of addition (the spacing
    # of float32 at 1e8 is 8): ((1e8 + 1) - 1e8) + 1 = (1e8 - 1e8) + 1 = 1,
    # whereas pairs (1e8 + 1) + (-1e8 + 1) = 1e8 - 1e8 = 0, and the reverse
    # order ((1 - 1e8) + 1) + 1e8 = 0
    v = np.float32([[1e8], [1.0], [-1e8], [1.0]])
    assert Q.group_column_sum(v)[0] == np.float32(1.0)
    assert Q.group_column_sum(v[::-1])[0] == np.float32(0.0)
    # 20 slots (more than one 16-slot chunk): a chunked sum would give 0 here
    w = np.zeros((20, 1), np.float32)
    w[0], w[1], w[16], w[17] = 1e8, 1.0, -1e8, 1.0
    assert Q.group_column_sum(w)[0] == np.float32(1.0)


# ---------------------------------------------------------------------------
# App. D grouping: pins against explicit matrices and brute force
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("k", [1, 2, 8, 64])
def test_bhq_scale_norm_is_the_explicit_bound(k):
    # |S^-1|_F^2 from the plan's scalars equals the Frobenius norm of the
    # explicit inverse blocks diag(d)^-1 H (theory module, Eq. matrix-quantizer-variance)
    rng = np.random.default_rng(k)
    x = (rng.lognormal(0, 2, (200, 1)) * rng.standard_normal((200, 48))).astype(np.float32)
    q = Q.quantize_bhq(x, 5, k, seed=0, stream=1)
    D = x.shape[1]
    assert Q.bhq_scale_norm(q["plan"]) == pytest.approx(4.0 / D * theory.matrix_var_bound(q, D), rel=1e-12)


def explicit_inverse_norm(plan):
    """|S^-1|_F^2 by inverting the explicit N x N block-diagonal scale matrix
    S = blockdiag(H_g diag(d_g)) of a plan (numpy's LU inverse)."""
    N = len(plan["perm"])
    S = np.zeros((N, N))
    for info in plan["groups"]:
        b, kg = info["base"], info["size"]
        d = plan["scale"][b: b + kg].astype(np.float64)
        Hk = theory.householder_matrix(kg) if kg > 1 else np.eye(1)
        S[b: b + kg, b: b + kg] = Hk @ np.diag(d)
    return float((np.linalg.inv(S) ** 2).sum())


def tiny_cases():
    rng = np.random.default_rng(21)
    cases = []
    for n in range(1, 9):
        for t in range(3):
            x = (rng.lognormal(0, 2, (n, 1)) * rng.standard_normal((n, 5))).astype(np.float32)
            cases.append(x)
    x = (0.01 * rng.standard_normal((8, 5))).astype(np.float32)
    x[3] = 50 * rng.standard_normal(5)                 # one outlier
    cases.append(x)
    x = rng.standard_normal((7, 4)).astype(np.float32)
    x[[1, 4]] = x[0]                                   # tied norms
    cases.append(x)
    return cases


def exact_counts(M_sorted, G):
    """App. D's cumulative rounding in exact rational arithmetic: the first i
    groups take round((N - G) P_i / P_G) small rows (None near a half-integer)."""
    N = len(M_sorted)
    P = [Fraction(0)]
    for m in M_sorted:
        P.append(P[-1] + Fraction(float(m)))
    out, prev = [], 0
    for i in range(1, G + 1):
        q = Fraction(N - G) * P[i] / P[G] if P[G] > 0 else Fraction((N - G) * i, G)
        frac = q - math.floor(q)
        if abs(frac - Fraction(1, 2)) < Fraction(1, 10 ** 9):
            return None
        c = math.floor(q + Fraction(1, 2))
        out.append(c - prev)
        prev = c
    return out


def test_appd_counts_are_the_proportional_cumulative_rounding():
    for x in tiny_cases() + [heavy_rows(22, 60, 3)]:
        N = x.shape[0]
        M = np.abs(x).max(axis=1)
        Ms = np.sort(M)[::-1]
        P = Q.appd_prefix(Ms)
        for G in range(1, N + 1):
            n = Q.appd_small_counts(P, N, G)
            assert len(n) == G and min(n) >= 0 and sum(n) == N - G
            ref = exact_counts(Ms, G)
            if ref is not None:
                assert n == ref, (N, G, n, ref)


def test_appd_objective_is_the_explicit_inverse_norm():
    # for every G, the objective App. D scores equals |S^-1|_F^2 of the plan
    # it builds, with S assembled explicitly and inverted
    for x in tiny_cases():
        N = x.shape[0]
        _, obj = Q.bhq_appd(x, 4)
        for G in range(1, N + 1):
            plan = Q.bhq_appd_plan(x, 4, G)
            assert plan["G"] == G
            assert obj[G - 1] == pytest.approx(explicit_inverse_norm(plan), rel=1e-11)


def compositions(total, parts):
    if parts == 1:
        yield (total,)
        return
    for first in range(total + 1):
        for rest in compositions(total - first, parts - 1):
            yield (first,) + rest


def test_appd_choice_brute_force_over_contiguous_groupings():
    # every contiguous grouping (G large rows, then n_1..n_G small rows in
    # sorted order) of N <= 7 rows, scored by the explicit inverse: App. D's
    # candidate for each G is one of them, and its choice is the best of its
    # candidates; PSQ (G = N) and one group (G = 1) are candidates, so the
    # choice never loses to either
    for x in [c for c in tiny_cases() if c.shape[0] <= 7]:
        N = x.shape[0]
        _, _, M, order = Q._sorted_rows(x)
        G_best, obj = Q.bhq_appd(x, 4)
        brute = {}
        for G in range(1, N + 1):
            for n in compositions(N - G, G):
                plan = Q._build_plan(x, 4, order, Q.appd_members(order, G, list(n)))
                brute[(G, n)] = explicit_inverse_norm(plan)
        cands = {}
        for G in range(1, N + 1):
            n = tuple(Q.appd_small_counts(Q.appd_prefix(M[order]), N, G))
            cands[G] = brute[(G, n)]
            assert obj[G - 1] == pytest.approx(cands[G], rel=1e-11)
        best = min(cands.values())
        assert cands[G_best] == pytest.approx(best, rel=1e-11)
        assert all(cands[G] > best * (1 + 1e-9) for G in range(1, G_best))   # ties go to fewer groups
        assert cands[G_best] <= cands[N] * (1 + 1e-12) and cands[G_best] <= cands[1] * (1 + 1e-12)
        assert min(brute.values()) <= cands[G_best] * (1 + 1e-12)


def test_appd_equal_norms_give_the_fixed_block_plan():
    # every row with the same infinity norm: App. D's proportional sizes are
    # equal, so for N = G k its plan for G is the fixed-block plan of size k
    rng = np.random.default_rng(23)
    for N, k in ((12, 3), (64, 8), (40, 5)):
        x = rng.uniform(-1, 1, (N, 9)).astype(np.float32)
        x[:, 0] = 2.0                                   # M = 2 for every row
        G = N // k
        a = Q.bhq_appd_plan(x, 5, G)
        b = Q.bhq_plan(x, 5, k)
        np.testing.assert_array_equal(a["perm"], b["perm"])
        np.testing.assert_array_equal(a["group_off"], b["group_off"])
        np.testing.assert_array_equal(a["scale"], b["scale"])
        np.testing.assert_array_equal(a["zero"], b["zero"])


def test_appd_literal_estimate_always_picks_one_group():
    # App. D's approximation sum_i M_i^2 / ((N - G) M_i / S_G) = S_G^2 / (N - G)
    # grows with G: read literally the search always ends at G = 1
    rng = np.random.default_rng(24)
    M = np.sort(rng.lognormal(0, 2, 50))[::-1]
    est = []
    for G in range(1, 50):
        S = M[:G].sum()
        lit = sum(m * m / ((50 - G) * m / S) for m in M[:G])
        assert lit == pytest.approx(S * S / (50 - G), rel=1e-12)
        est.append(lit)
    assert all(b > a for a, b in zip(est, est[1:]))


def test_appd_equal_rows_keep_per_row_scales():
    # identical rows: lambda2 = 2 max|row| >= lambda1 = R, so any group costs
    # more than its rows do alone (App. C.4): every row is its own group (PSQ)
    rng = np.random.default_rng(3)
    x = np.tile(rng.standard_normal((1, 40)).astype(np.float32), (130, 1))
    G, obj = Q.bhq_appd(x, 5)
    assert G == 130
    B = Q.n_bins(5)
    R = float(x[0].max() - x[0].min())
    assert obj[-1] == pytest.approx(130 * (R / B) ** 2, rel=1e-6)


def test_appd_spreads_a_single_outlier():
    # one row 1e8 times larger than the rest: one group of all the rows, whose
    # bound ~ lambda1^2 / (B^2 N) beats the per-row lambda1^2 / B^2 (Sec. 4.2)
    rng = np.random.default_rng(4)
    x = (1e-4 * rng.standard_normal((64, 32))).astype(np.float32)
    x[9] = (1e4 * rng.standard_normal(32)).astype(np.float32)
    G, obj = Q.bhq_appd(x, 5)
    assert G == 1
    assert obj[0] < obj[-1] / 32


def test_appd_zero_matrix_ties_to_one_group():
    # unit scales everywhere: |S^-1|_F^2 = N for every G, and ties go to fewer groups
    G, obj = Q.bhq_appd(np.zeros((30, 8), np.float32), 4)
    assert all(v == 30.0 for v in obj)
    assert G == 1


def test_appd_quantizer_is_unbiased_within_its_bound():
    x = heavy_rows(25, 150, 20)
    q = Q.quantize_bhq(x, 5, 0, seed=2, stream=1)
    assert q["k"] == 0 and q["G"] == Q.bhq_appd(x, 5)[0]
    np.testing.assert_array_equal(q["code"], Q.quantize_bhq(x, 5, 0, seed=2, stream=1, plan=q["plan"])["code"])
    m = theory.exact_mean(x, q)
    for g in q["plan"]["groups"]:
        mem = g["members"]
        assert np.abs(m[mem] - x[mem]).max() <= 2.0 ** -18 * np.abs(x[mem]).max()
    v = theory.exact_quantizer_variance(x, q)
    assert v <= x.shape[1] / 4.0 * Q.bhq_scale_norm(q["plan"]) * (1 + 1e-9)
    assert v < theory.exact_quantizer_variance(x, Q.quantize_psq(x, 5))
    y = theory.transformed_values(x, q)
    B = Q.n_bins(5)
    assert y.min() >= -1e-4 * B and y.max() <= B * (1 + 1e-4)
