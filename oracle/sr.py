"""Stochastic rounding SR(.) (oracle; test infrastructure only).

Sec. 3.3 defines SR(x) = ceil(x) with probability x - floor(x), floor(x)
otherwise.  A machine draw has finitely many bits, so the contract fixes a
24-bit uniform u = (32-bit Philox word) & 0xFFFFFF (its low 24 bits) and rounds up iff

    float(u) < frac * 2^24,   frac = y - floor(y)   (float32, exact for y >= 0)

which rounds up with probability ceil(frac * 2^24) / 2^24.  For y >= 0.5 every
float32 frac is a multiple of 2^-24, so this equals frac exactly and SR is
exactly unbiased there; below 0.5 the excess is under 2^-24 of a bin.

The quantizers clamp the rounded code to [0, B] (B = 2^b - 1, Sec. 3.3).
"""
import numpy as np

from . import philox

TWO24 = np.float32(16777216.0)


def uniform24(elem_index, seed, stream):
    """The 24-bit integer uniforms u in [0, 2^24) for the given element indices."""
    return (philox.draws(elem_index, seed, stream) & np.uint64(0xFFFFFF)).astype(np.int64)


def round_stochastic(y, u, B):
    """SR of float32 values `y` with 24-bit uniforms `u`; codes clamped to [0, B]."""
    y = np.asarray(y, dtype=np.float32)
    fl = np.floor(y).astype(np.float32)
    frac = (y - fl).astype(np.float32)
    up = np.asarray(u, dtype=np.int64).astype(np.float32) < (frac * TWO24).astype(np.float32)
    code = fl.astype(np.float64) + up.astype(np.float64)
    return np.clip(code, 0, B).astype(np.int64)


def round_nearest_even(y, B):
    """Deterministic rounding used by Q_f and Q_theta (ties to even), clamped to [0, B]."""
    y = np.asarray(y, dtype=np.float32)
    return np.clip(np.rint(y).astype(np.float64), 0, B).astype(np.int64)


def round_up_probability(y):
    """Exact probability that SR rounds float32 `y` up under the 24-bit contract."""
    y = np.asarray(y, dtype=np.float32)
    fl = np.floor(y).astype(np.float32)
    frac = (y - fl).astype(np.float32).astype(np.float64)
    return np.ceil(frac * 2.0 ** 24) / 2.0 ** 24


def exact_mean_code(y, B):
    """E[code] of SR on float32 `y` before the clamp matters (0 <= y <= B)."""
    y = np.asarray(y, dtype=np.float32)
    return np.floor(y).astype(np.float64) + round_up_probability(y)


def exact_var_code(y):
    """Var[code] = p (1 - p) (App. C, variance of stochastic rounding)."""
    p = round_up_probability(y)
    return p * (1.0 - p)
