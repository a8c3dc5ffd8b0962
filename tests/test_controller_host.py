"""Host logic of the reward-coordinated controller (no GPU): retention per
Eq. 1 over the reward history, the S-token compression trigger, length
bookkeeping by the kept-count rule, and the two-top-band probe trigger."""
import numpy as np
import pytest

import oracle
from paper_2608_04771_amd.controller import RecoPolicy, RewardSchedule


def test_eq1_retention_follows_reward_history():
    pol = RecoPolicy(retention="eq1", lam=0.25, delta=0.1, window=32)
    s = RewardSchedule(pol, prompt_len=512)
    rng = np.random.default_rng(0)
    hist = []
    for i in range(40):
        s.token_appended(int(rng.integers(1, 400)))
        v = float(rng.beta(2, 5))
        hist.append(v)
        compress, r, _ = s.end_step(v)
        assert compress
        assert r == pytest.approx(oracle.retention_eq1(hist, 0.25, 0.1), abs=1e-15)
        assert 0.15 - 1e-15 <= r <= 0.35 + 1e-15
        L_before = s.length
        s.compressed(r)
        assert s.length == oracle.kept_count(L_before, 32, r)


def test_clamp_retention_and_interval_trigger():
    pol = RecoPolicy(retention="clamp", window=16, interval=100)
    s = RewardSchedule(pol, prompt_len=200)
    s.token_appended(60)
    compress, r, _ = s.end_step(0.5)
    assert not compress and r == 0.75                       # grown by 60 < S = 100
    s.token_appended(40)
    compress, r, _ = s.end_step(0.2)
    assert compress and r == 0.9                            # grown by 100 >= S
    s.compressed(r)
    assert s.length == oracle.kept_count(300, 16, 0.9) == 270
    assert s.length_at_compress == 270
    s.token_appended(99)
    assert not s.end_step(1.0)[0]
    s.token_appended(1)
    compress, r, _ = s.end_step(1.0)
    assert compress and r == 0.5


def test_probe_needs_two_consecutive_top_band_rewards():
    pol = RecoPolicy(tau_hi=0.8)
    s = RewardSchedule(pol, prompt_len=10)
    flags = []
    for v in [0.9, 0.5, 0.85, 0.8, 0.95, 0.79, 0.8, 0.8]:
        s.token_appended()
        flags.append(s.end_step(v)[2])
    assert flags == [False, False, False, True, True, False, False, True]


def test_steady_state_cache_length():
    """Compressing to r*L every S tokens converges to L* ~ r*S/(1-r)."""
    pol = RecoPolicy(retention="clamp", window=32, interval=200)
    s = RewardSchedule(pol, prompt_len=512)
    for _ in range(200):
        s.token_appended(200)
        compress, r, _ = s.end_step(0.3)                    # r = 0.85
        assert compress
        s.compressed(r)
    assert abs(s.length - 0.85 * 200 / 0.15) <= 2


def test_delta_zero_is_the_uniform_retention_ablation():
    pol = RecoPolicy(retention="eq1", lam=0.25, delta=0.0, window=32)
    s = RewardSchedule(pol, prompt_len=512)
    for v in np.random.default_rng(1).beta(2, 5, size=30):
        s.token_appended(100)
        compress, r, _ = s.end_step(float(v))
        assert compress and r == 0.25
        s.compressed(r)


def test_per_layer_lengths_follow_the_layer_budgets():
    NL = 6
    pol = RecoPolicy(retention="clamp", window=16, layer_spread=0.5)
    s = RewardSchedule(pol, prompt_len=1000, n_layers=NL)
    ref = [1000] * NL
    rng = np.random.default_rng(2)
    for _ in range(12):
        n = int(rng.integers(10, 300))
        s.token_appended(n)
        v = float(rng.uniform())
        compress, r, _ = s.end_step(v)
        assert compress and r == oracle.retention_from_reward(v)
        s.compressed(r)
        ref = [oracle.kept_count(L + n, 16, oracle.layer_retention(r, l, NL, 0.5)) for l, L in enumerate(ref)]
        assert s.lengths == ref
    assert s.lengths[0] > s.lengths[-1]                      # deeper layers keep less
    assert s.length == s.lengths[0] == s.length_at_compress
