"""Pins for the oracle's random stream and stochastic rounding.

* Philox4x32 against rocRAND's independent implementation (a different
  code base built here from its installed header): its ten-round generator,
  and seven of its rounds composed from its own round and key-bump functions
  (the FQT stream's count);
* statistical sanity of the 24-bit uniforms;
* SR: exact round-up probability (Sec. 3.3), variance p(1-p) (App. C), and
  brute-force enumeration of every outcome on tiny inputs.
"""
import itertools
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import philox, sr

ROCRAND_HDR = "/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"

ROCRAND_PROBE = r"""
#include <cstdio>
// the round and key-bump helpers are private members; open them for this probe
#define private public
#include <rocrand/rocrand_philox4x32_10.h>
#undef private
struct Eng : rocrand_device::philox4x32_10_engine {
  uint4 run(uint4 c, uint2 k) { return ten_rounds(c, k); }
  uint4 run7(uint4 c, uint2 k) {
    for (int r = 0; r < 6; ++r) { c = single_round(c, k); k = bumpkey(k); }
    return single_round(c, k);
  }
};
int main(int argc, char**) {
  Eng eng; unsigned c[4], k[2];
  while (scanf("%u %u %u %u %u %u", &c[0], &c[1], &c[2], &c[3], &k[0], &k[1]) == 6) {
    const uint4 ci{c[0], c[1], c[2], c[3]};
    const uint2 ki{k[0], k[1]};
    uint4 r = argc > 1 ? eng.run7(ci, ki) : eng.run(ci, ki);
    printf("%u %u %u %u\n", r.x, r.y, r.z, r.w);
  }
}
"""


@pytest.mark.skipif(not (os.path.exists(ROCRAND_HDR) and shutil.which("g++")),
                    reason="rocRAND header or g++ not available")
def test_philox_matches_rocrand(tmp_path):
    src = tmp_path / "p.cpp"
    src.write_text(ROCRAND_PROBE)
    exe = tmp_path / "p"
    subprocess.run(["g++", "-O1", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", str(src), "-o", str(exe)],
                   check=True, capture_output=True)
    rng = np.random.default_rng(7)
    cases = rng.integers(0, 2 ** 32, size=(500, 6), dtype=np.uint64)
    cases[0] = 0
    cases[1] = 2 ** 32 - 1
    inp = "\n".join(" ".join(str(int(v)) for v in row) for row in cases) + "\n"
    for rounds, args in ((10, []), (7, ["7"])):
        out = subprocess.run([str(exe)] + args, input=inp, capture_output=True, text=True, check=True).stdout
        ref = np.array([[int(t) for t in line.split()] for line in out.strip().splitlines()], dtype=np.uint64)
        got = np.stack(philox.philox4x32(cases[:, 0], cases[:, 1], cases[:, 2], cases[:, 3],
                                          cases[:, 4], cases[:, 5], rounds=rounds), axis=1)
        np.testing.assert_array_equal(got, ref)
    assert philox.ROUNDS == 7


def test_draw_counter_mapping():
    # element e uses word e & 3 of the block at counter e >> 2 (stream in word 2)
    e = np.arange(64, dtype=np.uint64)
    d = philox.draws(e, seed=0x123456789ABCDEF, stream=1)
    for blk in range(16):
        o = philox.philox4x32(blk, 0, 1, 0, 0x89ABCDEF, 0x1234567)
        for w in range(4):
            assert int(d[4 * blk + w]) == int(o[w])
    assert not np.array_equal(philox.draws(e, 0, 0), philox.draws(e, 0, 1))
    assert not np.array_equal(philox.draws(e, 0, 0), philox.draws(e, 1, 0))


def test_uniform24_statistics():
    u = sr.uniform24(np.arange(1 << 18, dtype=np.uint64), seed=3, stream=0)
    assert u.min() >= 0 and u.max() < (1 << 24)
    hist = np.bincount((u >> 16).astype(np.int64), minlength=256)
    expected = len(u) / 256
    chi2 = float(((hist - expected) ** 2 / expected).sum())
    assert chi2 < 350          # 255 dof: mean 255, sd ~22.6
    x = u.astype(np.float64) / 2 ** 24
    assert abs(x.mean() - 0.5) < 4 * np.sqrt(1 / 12 / len(x))
    # neighbouring draws are uncorrelated
    r = np.corrcoef(x[:-1], x[1:])[0, 1]
    assert abs(r) < 4 / np.sqrt(len(x))


def test_round_up_probability_is_frac_above_half():
    rng = np.random.default_rng(0)
    y = rng.uniform(0.5, 255, 10000).astype(np.float32)
    p = sr.round_up_probability(y)
    frac = y.astype(np.float64) - np.floor(y.astype(np.float64))
    np.testing.assert_array_equal(p, frac)
    # below one half the excess is under 2^-24
    y = rng.uniform(0, 0.5, 10000).astype(np.float32)
    p = sr.round_up_probability(y)
    d = p - y.astype(np.float64)
    assert (d >= 0).all() and (d < 2.0 ** -24).all()


def test_round_stochastic_against_threshold_definition():
    # every u below ceil(frac * 2^24) rounds up, every other u rounds down
    y = np.float32(3.25)
    t = 4194304                 # 0.25 * 2^24
    u = np.array([0, t - 1, t, t + 1, (1 << 24) - 1])
    c = sr.round_stochastic(np.full(5, y), u, 255)
    np.testing.assert_array_equal(c, [4, 4, 3, 3, 3])
    # integers never round up; the clamp holds the ends
    np.testing.assert_array_equal(sr.round_stochastic(np.float32([0, 7, 255]), [0, 0, 0], 255), [0, 7, 255])
    np.testing.assert_array_equal(sr.round_stochastic(np.float32([-0.5, 255.5]), [0, 0], 255), [0, 255])


def test_sr_variance_closed_form():
    # App. C: Var[SR(x)] = p (1 - p) <= 1/4
    y = np.float32([0.5, 1.25, 2.75, 3.0])
    np.testing.assert_allclose(sr.exact_var_code(y), [0.25, 0.1875, 0.1875, 0.0])


def test_sr_brute_force_moments():
    # enumerate both outcomes of every element of a 2 x 3 matrix: the joint
    # law's mean and total variance equal the closed forms
    y = np.float32([[0.75, 1.5, 2.125], [0.625, 3.0, 1.875]]).ravel()
    p = sr.round_up_probability(y)
    fl = np.floor(y).astype(np.float64)
    mean = np.zeros_like(fl)
    second = np.zeros_like(fl)
    for bits in itertools.product([0, 1], repeat=y.size):
        b = np.array(bits, np.float64)
        prob = float(np.prod(np.where(b == 1, p, 1 - p)))
        mean += prob * (fl + b)
        second += prob * (fl + b) ** 2
    np.testing.assert_allclose(mean, sr.exact_mean_code(y, 255), rtol=0, atol=1e-15)
    np.testing.assert_allclose((second - mean ** 2).sum(), sr.exact_var_code(y).sum(), atol=1e-12)


def test_sr_monte_carlo_matches_probability():
    y = np.float32(np.full(200000, 5.3))
    e = np.arange(y.size, dtype=np.uint64)
    c = sr.round_stochastic(y, sr.uniform24(e, 11, 1), 255)
    p = sr.round_up_probability(y[:1])[0]
    phat = (c == 6).mean()
    assert set(np.unique(c)) <= {5, 6}
    assert abs(phat - p) < 5 * np.sqrt(p * (1 - p) / y.size)
