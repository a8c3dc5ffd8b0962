"""Pins of the oracle's penalised sampling: the counter-based generator against
its published known-answer vectors, the Gumbel noise against its moments, the
greedy choice against a plain argmax, and the sampled distribution against
softmax(z~ / T) (Section 3.3: sample from the softmax of the penalised logits)."""
import json
import math
import os

import numpy as np
import pytest
import scipy.special
import scipy.stats

import oracle.reco_oracle as ro

HERE = os.path.dirname(os.path.abspath(__file__))


def test_philox_known_answer_vectors():
    kat = json.load(open(os.path.join(HERE, "golden", "philox4x32_10_kat.json")))
    for vec in kat["vectors"]:
        ctr = [np.uint64(int(x, 16)) for x in vec["counter"]]
        key = tuple(int(x, 16) for x in vec["key"])
        out = [int(x) for x in ro.philox4x32_10(ctr, key)]
        assert out == [int(x, 16) for x in vec["output"]]


def test_uniform_grid_is_open_and_symmetric():
    x = np.array([0, 1, 511, 512, 0x7FFFFFFF, 0x80000000, 0xFFFFFE00, 0xFFFFFFFF], dtype=np.uint32)
    u = ro.uniform_from_bits(x)
    assert u.dtype == np.float32
    assert u[0] == 2.0 ** -24 and u[-1] == 1 - 2.0 ** -24          # cell midpoints at both ends
    assert u[1] == u[2] == u[0] and u[3] == 3 * 2.0 ** -24           # 2^23 cells of width 2^-23
    assert (u > 0).all() and (u < 1).all()
    rng = np.random.default_rng(3)
    y = rng.integers(0, 2 ** 32, size=100000, dtype=np.uint64).astype(np.uint32)
    np.testing.assert_array_equal(ro.uniform_from_bits(y) + ro.uniform_from_bits(~y), np.float32(1.0))
    assert np.isfinite(-np.log(-np.log(ro.uniform_from_bits(x)))).all()


def test_gumbel_noise_moments():
    g = ro.gumbel_noise(3, 400000, seed=12345, offset=7).astype(np.float64)
    assert np.isfinite(g).all()
    assert abs(g.mean() - np.euler_gamma) < 0.01                  # E[G] = Euler-Mascheroni constant
    assert abs(g.var() - math.pi ** 2 / 6) < 0.03                 # Var[G] = pi^2 / 6
    ks = scipy.stats.kstest(g, scipy.stats.gumbel_r.cdf)
    assert ks.pvalue > 1e-3


def test_gumbel_noise_depends_on_row_seed_and_offset():
    a = ro.gumbel_noise(0, 64, 1, 0)
    assert not np.array_equal(a, ro.gumbel_noise(1, 64, 1, 0))
    assert not np.array_equal(a, ro.gumbel_noise(0, 64, 2, 0))
    assert not np.array_equal(a, ro.gumbel_noise(0, 64, 1, 1))
    assert np.array_equal(a, ro.gumbel_noise(0, 64, 1, 0))


def test_greedy_is_argmax_of_penalised_logits():
    rng = np.random.default_rng(0)
    z = (3 * rng.standard_normal((4, 500))).astype(np.float32)
    R = [7, 300, 499]
    z[:, 300] = 50.0                                             # a reflection token dominates the raw row
    v = np.array([0.1, 0.5, 0.9, 0.95], dtype=np.float32)
    zp, tok, _ = ro.penalty_sample(z, R, v, 0.4, 0.8, 0.0, 100.0, 100.0, 0.0, 0, 0)
    assert tok[0] == 300                                          # low band: no penalty
    for b in (1, 2, 3):
        assert tok[b] == int(np.argmax(np.where(np.isin(np.arange(500), R), z[b] - 100.0, z[b])))
        assert tok[b] != 300
    z2 = np.zeros((1, 10), dtype=np.float32)
    assert ro.penalty_sample(z2, [], [0.0], 0.4, 0.8, 0, 0, 0, 0.0, 0, 0)[1][0] == 0   # ties: lowest index


def test_sampling_distribution_is_softmax_of_penalised_logits():
    z = np.array([[1.0, 2.0, 0.5, 2.0, -1.0, 3.0]], dtype=np.float32)
    R = [5]
    T = 0.7
    counts = np.zeros(6)
    n = 20000
    for off in range(n):
        counts[ro.penalty_sample(z, R, [0.9], 0.4, 0.8, 0.0, 1.0, 2.0, T, 99, off)[1][0]] += 1
    zp = z[0].astype(np.float64).copy()
    zp[5] -= 2.0
    p = scipy.special.softmax(zp / T)
    chi2 = ((counts - n * p) ** 2 / (n * p)).sum()
    assert chi2 < scipy.stats.chi2.ppf(0.999, df=5), (counts / n, p)
