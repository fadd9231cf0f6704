"""Gradient, activation and weight quantizers (oracle; test infrastructure only).

Paper: Chen et al. 2020, "A Statistical Framework for Low-bitwidth Training of
Deep Neural Networks".

* PTQ, per-tensor quantizer, Sec. 3.3: Q(X) = SR(s (X - z)) / s + z with
  z = min X, s = B / R(X), R(X) = max X - min X, B = 2^b - 1.  The deterministic
  variant (nearest rounding) is the Q_f / Q_theta of App. E.
* PSQ, per-sample quantizer, Sec. 4.1 and App. C.3: the same per row i with
  s_i = B / R(row i) (the optimum of the per-sample problem); z_i = row min.
* BHQ, block Householder quantizer, Sec. 4.2, App. C.4 and App. D: rows sorted
  by their infinity norm; each group holds one large row and k-1 small rows;
  the group's scale block is Q diag(s1, s2, ..., s2) with Q the Householder
  reflection whose normal is 1/sqrt(k) - e_1, and s1, s2 the closed form of
  App. C.4.

Readings where the paper is silent (each is listed with its reason in the
design notes of the repository):
  * R = 0 gives s = 1; B/R beyond the float32 range saturates at FLT_MAX;
  * a rounded code is clamped to [0, B];
  * PSQ zero point is the row minimum (by analogy with PTQ);
  * BHQ with a fixed block size k: G = ceil(N/k) groups; group g takes the
    g-th largest row plus the next k-1 rows of the sorted tail, in order;
  * BHQ with adaptive groups (App. D, step 2): every number of groups G from
    1 to N is tried; group i takes the i-th largest row plus n_i small rows,
    n_i proportional to M_i with cumulative rounding (appd_small_counts),
    small rows in sorted order; each candidate is scored by the exact
    |S^-1|_F^2 of the plan it builds and the least wins (ties: fewer groups);
  * BHQ zero point: one offset c_g per group in the transformed domain,
    c_g = alpha s1 min(large row) - lambda2 s2 sqrt(k) / 2, which App. C.4's
    range bound places at the bottom of the transformed values;
  * lambda1 = 0 takes lambda2; lambda2 = 0 gives s2 = s1 = B sqrt(k)/lambda1;
    both zero give s1 = s2 = 1; a one-row group is a PSQ row;
  * cube roots are correctly rounded float32; the group column sum adds the
    group's slots one at a time in slot order (float32).

Offset codes (what the int8 contractions consume) are code - 2^(b-1).
"""
from fractions import Fraction
import math

import numpy as np

from . import sr

FLT_MAX = float(np.finfo(np.float32).max)


def n_bins(bits):
    """B = 2^b - 1 (Sec. 3.3)."""
    return (1 << int(bits)) - 1


def offset(bits):
    return 1 << (int(bits) - 1)


def to_f32_sat(v):
    """Round a float64 to float32 (nearest even), saturating at FLT_MAX."""
    f = np.float32(v)
    if not np.isfinite(f):
        f = np.float32(FLT_MAX)
    return f


def scale_from_range(R, B):
    """s = B / R in float32 (one correctly rounded division); R = 0 gives 1."""
    R = np.float32(R)
    if R == 0:
        return np.float32(1.0)
    with np.errstate(over="ignore"):
        s = np.float32(B) / R
    return s if np.isfinite(s) else np.float32(FLT_MAX)


def row_stats(x):
    """Per-row min, max, range R (float32 subtraction) and infinity norm M."""
    x = np.asarray(x, dtype=np.float32)
    mn = x.min(axis=1)
    mx = x.max(axis=1)
    R = (mx - mn).astype(np.float32)
    M = np.maximum(np.abs(mn), np.abs(mx)).astype(np.float32)
    return mn, mx, R, M


# ----------------------------------------------------------------------------
# PTQ and PSQ
# ----------------------------------------------------------------------------

def _affine_codes(x, s, z, bits, stochastic, seed, stream, elem_index):
    """y = s (x - z) in float32 (subtract, then multiply), then round."""
    B = n_bins(bits)
    t = (x - z).astype(np.float32)
    y = (s * t).astype(np.float32)
    if stochastic:
        u = sr.uniform24(elem_index, seed, stream)
        return sr.round_stochastic(y, u, B)
    return sr.round_nearest_even(y, B)


def quantize_ptq(x, bits, stochastic, seed=0, stream=0):
    """Per-tensor quantizer of Sec. 3.3 on a 2-D float32 array.

    Returns dict(code [rows, cols] int64 in [0, B], scale, zero, bits).  The
    element index of the SR draw is the logical row-major index i*cols + j.
    """
    x = np.asarray(x, dtype=np.float32)
    rows, cols = x.shape
    B = n_bins(bits)
    z = np.float32(x.min()) if x.size else np.float32(0)
    R = np.float32(np.float32(x.max()) - z) if x.size else np.float32(0)
    s = scale_from_range(R, B)
    e = np.arange(rows * cols, dtype=np.uint64).reshape(rows, cols)
    code = _affine_codes(x, s, z, bits, stochastic, seed, stream, e)
    return dict(kind="ptq", code=code, scale=np.float32(s), zero=np.float32(z), bits=int(bits))


def quantize_psq(x, bits, seed=0, stream=0):
    """Per-sample quantizer of Sec. 4.1: one (s_i, z_i) per row, SR per element."""
    x = np.asarray(x, dtype=np.float32)
    rows, cols = x.shape
    B = n_bins(bits)
    mn, _, R, _ = row_stats(x)
    s = np.array([scale_from_range(r, B) for r in R], dtype=np.float32)
    e = np.arange(rows * cols, dtype=np.uint64).reshape(rows, cols)
    code = _affine_codes(x, s[:, None], mn[:, None], bits, True, seed, stream, e)
    return dict(kind="psq", code=code, scale=s, zero=mn.astype(np.float32), bits=int(bits))


def shift_limit(bits):
    """E = min(4, 8 - b): the largest left shift that keeps a b-bit offset code
    (code - 2^(b-1) in [-2^(b-1), 2^(b-1) - 1]) inside int8."""
    return min(4, 8 - int(bits))


def quantize_shift(x, bits, seed=0, stream=0):
    """Per-tensor range with per-sample power-of-two steps (Sec. 4.3, the
    hardware variant of PSQ): R = max_i R_i, s = B / R; per row z_i = min_i,
    e_i = the largest e in [0, E] with R_i 2^e <= R, s_i = s 2^e_i (float32,
    saturating at FLT_MAX); y = s_i (x - z_i) with SR per element, as PSQ.

    `shift` holds E - e_i, the left shift that brings row i's offset codes to
    the common step 1 / (s 2^E).
    """
    x = np.asarray(x, dtype=np.float32)
    rows, cols = x.shape
    B = n_bins(bits)
    E = shift_limit(bits)
    mn, _, R, _ = row_stats(x)
    Rt = np.float32(R.max()) if rows else np.float32(0)
    st = scale_from_range(Rt, B)
    scale = np.zeros(rows, np.float32)
    shift = np.zeros(rows, np.int64)
    for i in range(rows):
        e = 0
        # R_i 2^(e+1) <= R: both sides exact (power-of-two scaling of a float32)
        while e < E and float(R[i]) * 2.0 ** (e + 1) <= float(Rt):
            e += 1
        scale[i] = to_f32_sat(float(st) * 2.0 ** e)
        shift[i] = E - e
    e_idx = np.arange(rows * cols, dtype=np.uint64).reshape(rows, cols)
    code = _affine_codes(x, scale[:, None], mn[:, None], bits, True, seed, stream, e_idx)
    return dict(kind="shift", code=code, scale=scale, zero=mn.astype(np.float32), shift=shift,
                step_scale=st, bits=int(bits))


def shifted_codes(q):
    """Offset codes shifted left by each row's shift: the int8 operands of the
    grad_W contraction for a `shift` quantizer (all rows at step 1 / (s 2^E))."""
    return offset_codes(q) << q["shift"][:, None]


def dequantize_affine(q):
    """Real value of each code, code / s + z, in float64 (Sec. 3.3 inverse map)."""
    s = np.asarray(q["scale"], dtype=np.float64)
    z = np.asarray(q["zero"], dtype=np.float64)
    if s.ndim == 1:
        s, z = s[:, None], z[:, None]
    return q["code"].astype(np.float64) / s + z


# ----------------------------------------------------------------------------
# BHQ
# ----------------------------------------------------------------------------

def cbrt_rn(x):
    """Correctly rounded float32 cube root of a non-negative finite float32.

    A float64 estimate picks a candidate; exact rational comparisons against
    the cubes of the midpoints to its float32 neighbours then move it to the
    nearest float32.  A midpoint has 25 significant bits, so its cube is never
    a float32 and ties cannot occur.
    """
    x = np.float32(x)
    if x == 0:
        return np.float32(0.0)
    X = Fraction(float(x))
    r = np.float32(np.cbrt(np.float64(x)))
    while True:
        up = np.nextafter(r, np.float32(np.inf))
        dn = np.nextafter(r, np.float32(0))
        mid_up = (Fraction(float(r)) + Fraction(float(up))) / 2
        mid_dn = (Fraction(float(r)) + Fraction(float(dn))) / 2
        if mid_up ** 3 < X:
            r = up
        elif mid_dn ** 3 > X:
            r = dn
        else:
            assert mid_up ** 3 != X and mid_dn ** 3 != X
            return np.float32(r)


def bhq_groups(N, k):
    """Row-slot layout of fixed-block BHQ: G = ceil(N/k) groups.

    Returns (G, sizes) with sizes[g] = 1 + the number of sorted-tail rows that
    group g takes (App. D builds groups of one large row plus small rows; the
    paper leaves the fixed-size assignment open: contiguous chunks of k-1).
    """
    G = -(-N // k)
    small = N - G
    sizes = []
    for g in range(G):
        lo = min(small, g * (k - 1))
        hi = min(small, (g + 1) * (k - 1))
        sizes.append(1 + hi - lo)
    return G, sizes


_cbrt_cache = {}


def _cbrt(v):
    """cbrt_rn, remembered per float32 value (the App. D search reuses them)."""
    key = float(v)
    r = _cbrt_cache.get(key)
    if r is None:
        r = _cbrt_cache[key] = float(cbrt_rn(np.float32(v)))
    return r


def group_scales(lam1, lam2, kg, B):
    """s1, s2 of a group of kg >= 2 rows (App. C.4), float32.

    s1 = B sqrt(k) / (a (a^2 + c^2 k)), s2 = B sqrt(k) / (c (a^2 + c^2 k)) with
    a = lambda1^(1/3), c = lambda2^(1/3): the closed form of App. C.4
    multiplied through by k^(1/3).  lambda1 = 0 takes lambda2; lambda2 = 0
    gives s1 = s2 = B sqrt(k) / lambda1; both zero give 1.  Returns
    (lambda1 as used, s1, s2, sqrt(k)).
    """
    lam1, lam2 = np.float32(lam1), np.float32(lam2)
    if lam1 == 0:
        lam1 = lam2
    sk = math.sqrt(float(kg))
    if lam1 == 0 and lam2 == 0:
        s1 = s2 = np.float32(1.0)
    elif lam2 == 0:
        s1 = s2 = to_f32_sat((float(B) * sk) / float(lam1))
    else:
        a = _cbrt(lam1)
        c = _cbrt(lam2)
        t = a * a + (c * c) * float(kg)
        num = float(B) * sk
        s1 = to_f32_sat(num / (a * t))
        s2 = to_f32_sat(num / (c * t))
    return lam1, s1, s2, sk


def group_term(s1, s2, kg):
    """A group's share of |S^-1|_F^2 (Eq. matrix-quantizer-variance): S^-1 of
    the group is diag(s1, s2, .., s2)^-1 times an orthogonal reflection, so
    1/s1^2 + (k_g - 1)/s2^2 (a one-row group: 1/s^2), in float64."""
    s1 = float(s1)
    term = 1.0 / (s1 * s1)
    if kg > 1:
        s2 = float(s2)
        term = term + float(kg - 1) * (1.0 / (s2 * s2))
    return term


def _sorted_rows(x):
    """Row statistics and the order of Sec. 4.2 / App. D: M descending, ties by
    row index ascending."""
    mn, mx, R, M = row_stats(x)
    order = np.lexsort((np.arange(len(M)), -M))
    return mn, R, M, order


def _build_plan(x, bits, order, members_list):
    """Per-slot scales and zero points of a BHQ plan whose groups (each a list of
    original rows, large row first) are given in slot order."""
    x = np.asarray(x, dtype=np.float32)
    N, D = x.shape
    B = n_bins(bits)
    mn, mx, R, M = row_stats(x)
    perm, group_off = [], [0]
    scale = np.zeros(N, np.float32)
    zero = np.zeros(N, np.float32)
    groups = []
    for members in members_list:
        base = len(perm)
        perm.extend(members)
        group_off.append(len(perm))
        kg = len(members)
        info = dict(members=list(members), base=base, size=kg)
        if kg == 1:
            i = members[0]
            scale[base] = scale_from_range(R[i], B)
            zero[base] = mn[i]
        else:
            big = members[0]
            lam2 = np.float32(np.float32(2.0) * np.float32(M[members[1:]].max()))
            lam1, s1, s2, sk = group_scales(R[big], lam2, kg, B)
            alpha = np.float32(1.0 / sk)
            oma = np.float32(np.float32(1.0) - alpha)
            cg = np.float32(((float(alpha) * float(s1)) * float(mn[big]))
                            - (((0.5 * float(lam2)) * float(s2)) * sk))
            scale[base] = s1
            scale[base + 1: base + kg] = s2
            zero[base: base + kg] = cg
            info.update(lam1=lam1, lam2=lam2, s1=s1, s2=s2, alpha=alpha, oma=oma, cg=cg, sk=sk)
        groups.append(info)
    return dict(perm=np.array(perm, np.int64), group_off=np.array(group_off, np.int64),
                scale=scale, zero=zero, groups=groups, G=len(members_list), bits=int(bits), sorted=order)


def bhq_plan(x, bits, k):
    """Sort, grouping and per-group scalars of the block Householder quantizer
    with a fixed block size k >= 1.

    Sec. 4.2 / App. D: sort the row infinity norms M_i in descending order
    (ties: lower row index first); the first G = ceil(N/k) rows are the large
    rows; group g takes the g-th large row and the next k-1 rows of the sorted
    tail.  Scalars per group: group_scales.
    """
    x = np.asarray(x, dtype=np.float32)
    N = x.shape[0]
    order = _sorted_rows(x)[3]
    G, sizes = bhq_groups(N, k)
    members_list, t = [], G
    for g in range(G):
        members_list.append([int(order[g])] + [int(i) for i in order[t: t + sizes[g] - 1]])
        t += sizes[g] - 1
    plan = _build_plan(x, bits, order, members_list)
    plan["k"] = int(k)
    return plan


# ----------------------------------------------------------------------------
# App. D: adaptive grouping
# ----------------------------------------------------------------------------

def appd_prefix(M_sorted):
    """P_i = M_(1) + .. + M_(i) of the sorted infinity norms, float64, added one
    at a time in sorted order; P_0 = 0."""
    P = [0.0]
    for m in M_sorted:
        P.append(P[-1] + float(m))
    return P


def appd_small_counts(P, N, G):
    """Number of small rows n_1..n_G of each group for G groups (App. D, step 2).

    App. D sizes the i-th group's share of the N - G small rows in proportion
    to M_i: (N - G) M_i / sum_{j<=G} M_j, which is fractional.  Rounded
    cumulatively: with q_i = (N - G) P_i / P_G (float64: product, then
    quotient), the first i groups take c_i = floor(q_i + 1/2) small rows
    (c_G = N - G), so n_i = c_i - c_(i-1) >= 0 and the counts add up to N - G.
    If the G largest norms are all zero, P_i is replaced by i.
    """
    small = N - G
    S = P[G]
    counts, prev = [], 0
    for i in range(1, G + 1):
        if i == G:
            c = small
        else:
            q = (float(small) * P[i]) / S if S > 0 else float(small * i) / float(G)
            c = min(int(math.floor(q + 0.5)), small)
        counts.append(c - prev)
        prev = c
    return counts


def appd_members(order, G, counts):
    """Groups for G: group i is the i-th largest row, then its n_i small rows
    taken from the sorted tail in order."""
    members_list, t = [], G
    for i in range(G):
        members_list.append([int(order[i])] + [int(r) for r in order[t: t + counts[i]]])
        t += counts[i]
    return members_list


def appd_objective(R, M, order, P, bits, G):
    """|S^-1|_F^2 of the App. D plan with G groups: the sum over groups of
    group_term, float64, added in group order.  A group's lambda1 is its large
    row's range and lambda2 twice the largest infinity norm of its small rows
    (the first of them: they come in sorted order)."""
    N = len(order)
    B = n_bins(bits)
    counts = appd_small_counts(P, N, G)
    total, t = 0.0, G
    for i in range(G):
        big = order[i]
        n = counts[i]
        if n == 0:
            s = scale_from_range(R[big], B)
            term = group_term(s, s, 1)
        else:
            lam2 = np.float32(np.float32(2.0) * M[order[t]])
            _, s1, s2, _ = group_scales(R[big], lam2, n + 1, B)
            term = group_term(s1, s2, n + 1)
        total = total + term
        t += n
    return total


def bhq_appd(x, bits):
    """App. D, step 2: loop over the number of groups G = 1..N and keep the G
    whose plan has the least |S^-1|_F^2 (ties: the smaller G).

    App. D's own estimate of the objective, sum_i M_i^2 / ((N - G) M_i / sum M),
    equals (sum of the G largest M)^2 / (N - G), which grows with G, so read
    literally it always keeps one group; here every candidate is scored by the
    exact factor |S^-1|_F^2 of the variance bound (D/4)|S^-1|_F^2 (Eq.
    matrix-quantizer-variance) of the plan App. D's sizes build.
    Returns (G, [objective for G = 1..N]).
    """
    x = np.asarray(x, dtype=np.float32)
    N = x.shape[0]
    _, R, M, order = _sorted_rows(x)
    P = appd_prefix(M[order])
    obj = [appd_objective(R, M, order, P, bits, G) for G in range(1, N + 1)]
    best = 1
    for G in range(2, N + 1):
        if obj[G - 1] < obj[best - 1]:
            best = G
    return best, obj


def bhq_appd_plan(x, bits, G=None):
    """The App. D plan: G groups (bhq_appd's choice when G is None)."""
    x = np.asarray(x, dtype=np.float32)
    N = x.shape[0]
    if G is None:
        G = bhq_appd(x, bits)[0]
    _, R, M, order = _sorted_rows(x)
    counts = appd_small_counts(appd_prefix(M[order]), N, G)
    plan = _build_plan(x, bits, order, appd_members(order, G, counts))
    plan["k"] = 0
    return plan


def bhq_scale_norm(plan):
    """|S^-1|_F^2 of a BHQ plan, the factor of the variance bound (D/4)|S^-1|_F^2
    (Eq. matrix-quantizer-variance): group_term summed over groups in slot
    order, float64."""
    total = 0.0
    for info in plan["groups"]:
        base, kg = info["base"], info["size"]
        s2 = plan["scale"][base + 1] if kg > 1 else plan["scale"][base]
        total = total + group_term(plan["scale"][base], s2, kg)
    return total


# ----------------------------------------------------------------------------
# BHQ transform and quantizer
# ----------------------------------------------------------------------------

def group_column_sum(v):
    """Column sums of a group's scaled rows v [k_g, D], float32, adding the
    slots one at a time in slot order."""
    S = np.zeros(v.shape[1], np.float32)
    for p in range(v.shape[0]):
        S = (S + v[p]).astype(np.float32)
    return S


def bhq_transform(rows, info):
    """y' = Q diag(s1, s2..s2) G_g - c_g for one group, float32 (Sec. 4.2).

    v_p = d_p g_p; S = group column sum; tau = (alpha S - v_0) / (1 - alpha);
    Y_0 = v_0 + (1 - alpha) tau, Y_p = v_p - alpha tau; then subtract c_g.
    This is the reflection I - 2 n n^T / |n|^2 with n = alpha 1 - e_0 applied
    as a rank-1 update (|n|^2 = 2 (1 - alpha)).
    """
    kg = info["size"]
    d = np.array([info["s1"]] + [info["s2"]] * (kg - 1), np.float32)
    v = (d[:, None] * rows).astype(np.float32)
    S = group_column_sum(v)
    alpha, oma = np.float32(info["alpha"]), np.float32(info["oma"])
    m = (alpha * S).astype(np.float32)
    m = (m - v[0]).astype(np.float32)
    tau = (m / oma).astype(np.float32)
    Y = np.empty_like(v)
    Y[0] = (v[0] + (oma * tau).astype(np.float32)).astype(np.float32)
    if kg > 1:
        Y[1:] = (v[1:] - (alpha * tau).astype(np.float32)[None, :]).astype(np.float32)
    return (Y - np.float32(info["cg"])).astype(np.float32)


def quantize_bhq(x, bits, k, seed=0, stream=0, plan=None):
    """Block Householder quantizer (Sec. 4.2) with a fixed block size k >= 1, or
    with App. D's adaptive groups for k = 0.

    Codes are returned in slot order (group by group); the SR draw of slot p,
    column j uses element index perm[p] * cols + j (its original position).
    """
    x = np.asarray(x, dtype=np.float32)
    N, D = x.shape
    B = n_bins(bits)
    if plan is None:
        plan = bhq_appd_plan(x, bits) if k == 0 else bhq_plan(x, bits, k)
    code = np.zeros((N, D), np.int64)
    cols = np.arange(D, dtype=np.uint64)
    for info in plan["groups"]:
        mem = info["members"]
        base, kg = info["base"], info["size"]
        rows = x[mem]
        e = np.asarray(mem, dtype=np.uint64)[:, None] * np.uint64(D) + cols[None, :]
        if kg == 1:
            s, z = plan["scale"][base], plan["zero"][base]
            y = (s * (rows - z).astype(np.float32)).astype(np.float32)
        else:
            y = bhq_transform(rows, info)
        u = sr.uniform24(e, seed, stream)
        code[base: base + kg] = sr.round_stochastic(y, u, B)
    return dict(kind="bhq", code=code, scale=plan["scale"], zero=plan["zero"], perm=plan["perm"],
                group_off=plan["group_off"], bits=int(bits), plan=plan, k=plan["k"], G=plan["G"])


def dequantize_bhq(q):
    """Real values of a BHQ result in original row order, float64.

    Inverse map of Eq. (matrix-quantizer): G~_g = diag(d)^-1 Q (code + c_g),
    with the exact reflection (alpha = 1/sqrt(k_g) in float64); a one-row group
    is a PSQ row, code / s + z.
    """
    code = q["code"].astype(np.float64)
    N, D = code.shape
    out = np.zeros((N, D), np.float64)
    for info in q["plan"]["groups"]:
        base, kg, mem = info["base"], info["size"], info["members"]
        s = q["scale"][base: base + kg].astype(np.float64)
        z = q["zero"][base: base + kg].astype(np.float64)
        if kg == 1:
            out[mem[0]] = code[base] / s[0] + z[0]
            continue
        w = code[base: base + kg] + z[0]
        a = 1.0 / math.sqrt(kg)
        tau = (a * w.sum(axis=0) - w[0]) / (1.0 - a)
        Z = w - a * tau[None, :]
        Z[0] = w[0] + (1.0 - a) * tau
        out[mem] = Z / s[:, None]
    return out


def offset_codes(q):
    """Signed codes code - 2^(b-1), the int8 operands of the contractions."""
    return (q["code"] - offset(q["bits"])).astype(np.int64)


def dequantize(q):
    """Real values of any quantizer result, original row order, float64."""
    if q["kind"] == "bhq":
        return dequantize_bhq(q)
    return dequantize_affine(q)
