"""Pins of the oracle's policy variants (per-layer budgets, pooled scores):
closed forms, invariants and brute force on tiny inputs."""
import numpy as np
import pytest

import oracle.reco_oracle as ro


def test_layer_retention_single_level_when_spread_is_zero():
    for NL in (1, 2, 28, 64):
        for r in (0.15, 0.5, 1.0):
            assert all(ro.layer_retention(r, l, NL, 0.0) == r for l in range(NL))


def test_layer_retention_is_a_descending_line_with_mean_r():
    for NL, r, rho in [(28, 0.5, 0.5), (32, 0.3, 0.9), (2, 0.4, 0.25), (64, 0.25, 0.6)]:
        rl = np.array([ro.layer_retention(r, l, NL, rho) for l in range(NL)])
        assert rl[0] == pytest.approx(r * (1 + rho), rel=1e-15)          # most cache at the bottom
        assert rl[-1] == pytest.approx(r * (1 - rho), rel=1e-15)
        assert (np.diff(rl) < 0).all()
        np.testing.assert_allclose(np.diff(rl), np.diff(rl)[0], rtol=1e-12)   # equal steps
        assert rl.mean() == pytest.approx(r, rel=1e-14)                  # budget preserved on average


def test_layer_retention_cap_and_edges():
    rl = [ro.layer_retention(0.8, l, 5, 0.5) for l in range(5)]
    assert rl[0] == 1.0 and rl[1] == 1.0 and rl[2] == pytest.approx(0.8)  # 1.2 and 1.0 capped
    assert ro.layer_retention(0.7, 0, 1, 0.9) == 0.7
    with pytest.raises(ValueError):
        ro.layer_retention(0.5, 0, 4, 1.0)


def _pool_brute(s, L, w, k, mode):
    P = L - min(w, L)
    h = k // 2
    out = list(s[:L])
    for j in range(P):
        vals = [s[i] for i in range(P) if abs(i - j) <= h]
        out[j] = max(vals) if mode == "max" else sum(vals) / len(vals)
    return np.array(out)


@pytest.mark.parametrize("mode", ["max", "mean"])
def test_pool_matches_brute_force_on_tiny_inputs(mode):
    rng = np.random.default_rng(0)
    for L, w, k in [(10, 3, 3), (17, 4, 5), (9, 9, 3), (6, 1, 7), (40, 8, 11), (5, 8, 3), (1, 1, 1), (12, 2, 1)]:
        s = rng.exponential(size=L)
        np.testing.assert_allclose(ro.pool_scores(s, L, w, k, mode), _pool_brute(s, L, w, k, mode), rtol=1e-14)


def test_pool_kernel_one_is_identity_and_constant_stays_constant():
    s = np.random.default_rng(1).exponential(size=100)
    for mode in ("max", "mean"):
        np.testing.assert_array_equal(ro.pool_scores(s, 100, 16, 1, mode), s)
    c = np.full(64, 0.25)
    np.testing.assert_allclose(ro.pool_scores(c, 64, 8, 7, "mean"), c, rtol=1e-15)   # edges too
    np.testing.assert_array_equal(ro.pool_scores(c, 64, 8, 7, "max"), c)


def test_pool_max_spreads_a_spike_over_the_kernel_width():
    s = np.zeros(50)
    s[20] = 3.0
    out = ro.pool_scores(s, 50, 10, 7, "max")
    assert (out[17:24] == 3.0).all() and out[16] == 0 and out[24] == 0


def test_pool_mean_of_a_ramp_is_the_ramp_inside():
    s = np.arange(60, dtype=np.float64)
    out = ro.pool_scores(s, 60, 10, 9, "mean")
    np.testing.assert_allclose(out[4:46], s[4:46], rtol=1e-15)           # centred window of a line
    assert out[0] == pytest.approx(np.mean(s[0:5]))                     # shrinks at the prefix start
    assert out[49] == pytest.approx(np.mean(s[45:50]))                  # and stops at the window


def test_pool_leaves_the_window_alone_and_ignores_it():
    s = np.zeros(30)
    s[25] = 9.0                                                          # inside the window [22, 30)
    s[21] = 1.0                                                          # last prefix position
    for mode in ("max", "mean"):
        out = ro.pool_scores(s, 30, 8, 9, mode)
        np.testing.assert_array_equal(out[22:], s[22:])
        assert out[:22].max() <= 1.0                                     # the window spike does not leak


def test_compress_cache_takes_per_layer_retention():
    rng = np.random.default_rng(2)
    NL, B, H, L, D, w = 3, 2, 1, 50, 8, 4
    K = rng.standard_normal((NL, B, H, L, D))
    V = rng.standard_normal((NL, B, H, L, D))
    lens = np.full((NL, B, H), L)
    Q = rng.standard_normal((NL, B, 2, w, D))
    ret = [[ro.layer_retention(r, l, NL, 0.5) for r in (0.4, 0.6)] for l in range(NL)]
    _, idx, _, _, lens2 = ro.compress_cache(K, V, lens, Q, ret, w, 0.3)
    for l in range(NL):
        for b in range(B):
            assert lens2[l, b, 0] == ro.kept_count(L, w, ret[l][b])
    assert lens2[0, 0, 0] > lens2[2, 0, 0]
