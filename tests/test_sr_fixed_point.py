"""The 8.24 fixed-point form of the stochastic-rounding decision (used by the
device quantizers) against the oracle's float rule (Sec. 3.3 rounding with a
24-bit uniform), on the CPU.

With yc = clamp(y, 0, B), T = ceil(yc * 2^24) and u' = 2^24 - 1 - u, the
carry of T + u' into bit 24 must be set exactly when the oracle rounds up, and
(T + u' - half * 2^24) >> 24 must be the offset code.  The inputs include the
decision boundary itself: words whose 24-bit uniform is ceil(frac * 2^24) and
the one below it.
"""
import numpy as np
import pytest

from oracle import sr

F32 = np.float32


def fixed_point_codes(y, words, bits):
    """Offset codes from the fixed-point rule, evaluated in integers."""
    B = (1 << bits) - 1
    half = 1 << (bits - 1)
    yc = np.minimum(np.maximum(np.asarray(y, F32), F32(0)), F32(B)).astype(F32)
    t = np.ceil((yc * F32(16777216.0)).astype(F32)).astype(np.float64).astype(np.uint64)
    u_prime = ((words & np.uint32(0xFFFFFF)) ^ np.uint32(0xFFFFFF)).astype(np.uint64)
    acc = (t + u_prime - np.uint64(half << 24)) & np.uint64(0xFFFFFFFF)
    return acc.astype(np.uint32).view(np.int32) >> 24


@pytest.mark.parametrize("bits", [2, 4, 5, 8])
def test_fixed_point_equals_float_rule(bits):
    rng = np.random.default_rng(bits)
    B = (1 << bits) - 1
    n = 200_000
    fl = np.floor(rng.uniform(0, B, n))
    y = np.concatenate([
        rng.uniform(-2, B + 2, n),                                   # clamping on both sides
        rng.uniform(0, 1e-6, n),                                     # tiny fractions
        fl,                                                          # integers
        fl + rng.integers(0, 1 << 24, n) / 2.0 ** 24,                # fractions on the 2^-24 grid
        rng.uniform(0, 2.0 ** -20, n),                               # fractions below the grid
        np.array([0.0, B, np.nextafter(F32(B), F32(0)), 2.0 ** -24, 1 - 2.0 ** -24, 1e-45, np.inf, -np.inf]),
    ]).astype(F32)
    words = rng.integers(0, 1 << 32, y.size, dtype=np.uint64)
    # half the words sit on the decision boundary: u = ceil(frac * 2^24) or one below
    with np.errstate(invalid="ignore"):
        fr = np.nan_to_num((y - np.floor(y)).astype(F32) * F32(2 ** 24), nan=0.0, posinf=0.0, neginf=0.0)
    on_edge = rng.random(y.size) < 0.5
    u_edge = np.clip(np.ceil(fr[on_edge]) - rng.integers(0, 2, on_edge.sum()), 0, 2 ** 24 - 1).astype(np.uint64)
    words[on_edge] = u_edge | (rng.integers(0, 256, on_edge.sum(), dtype=np.uint64) << np.uint64(24))
    words = words.astype(np.uint32)
    with np.errstate(invalid="ignore"):
        ref = sr.round_stochastic(y, (words & np.uint32(0xFFFFFF)).astype(np.int64), B)
    got = fixed_point_codes(y, words, bits) + (1 << (bits - 1))
    assert np.array_equal(got, ref)
