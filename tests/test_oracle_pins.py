"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test checks one oracle function against a closed form, an invariant, a
special case that reduces to an independent library routine (scipy / torch
CPU), the paper's printed hyper-parameters, or exhaustive brute force on tiny
inputs.  ``test_oracle_mutants.py`` shows that plausible mistakes in the
oracle make these pins fail."""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.special
import torch
import torch.nn.functional as F

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


# ---------------------------------------------------------------- Eq. 1 / budget

def test_paper_hyperparameters_give_eq1_range():
    """Section 4.1 fixes lambda = 0.25 and delta = 0.1; Eq. 1 then keeps
    lambda_i inside [lambda - delta, lambda + delta] = [0.15, 0.35]."""
    hp = json.load(open(os.path.join(HERE, "golden", "paper_hyperparameters.json")))
    rng = np.random.default_rng(0)
    for _ in range(500):
        hist = rng.uniform(0, 1, size=rng.integers(1, 30))
        lam_i = oracle.retention_eq1(hist, hp["lambda"], hp["delta"])
        assert hp["lambda"] - hp["delta"] - 1e-15 <= lam_i <= hp["lambda"] + hp["delta"] + 1e-15


def test_eq1_closed_forms():
    # latest reward equal to the mean -> no adjustment
    assert oracle.retention_eq1([0.2, 0.6, 0.4], 0.25, 0.1) == pytest.approx(0.25, abs=1e-15)
    # all rewards equal -> base ratio
    assert oracle.retention_eq1([0.7, 0.7], 0.25, 0.1) == 0.25
    # history {0, 1}, latest 1: lambda - delta * (1 - 0.5) / 1 (high reward prunes harder)
    assert oracle.retention_eq1([0.0, 1.0], 0.25, 0.1) == pytest.approx(0.20, abs=1e-15)
    assert oracle.retention_eq1([1.0, 0.0], 0.25, 0.1) == pytest.approx(0.30, abs=1e-15)
    # the extremes of the history reach the bounds only when the mean sits at the other end
    assert oracle.retention_eq1([0.0, 0.0, 0.0, 1.0], 0.25, 0.1) == pytest.approx(0.25 - 0.1 * 0.75)


def test_default_retention_map_closed_form():
    assert oracle.retention_from_reward(0.0) == 1.0
    assert oracle.retention_from_reward(0.5) == 0.75
    assert oracle.retention_from_reward(1.0) == 0.5
    vs = np.linspace(0, 1, 101)
    rs = [oracle.retention_from_reward(v) for v in vs]
    assert all(a >= b for a, b in zip(rs, rs[1:]))          # higher reward keeps less


@pytest.mark.parametrize("L,w,r", [(2048, 32, 0.75), (16384, 64, 0.5), (1000, 32, 0.3),
                                   (7, 32, 0.5), (64, 64, 0.25), (100, 1, 1.0), (1, 1, 0.5),
                                   (1001, 32, 0.75), (16383, 64, 0.6), (2047, 32, 0.8133)])
def test_kept_count_is_exact_ceiling(L, w, r):
    exact = math.ceil(Fraction(r) * L)          # exact rational ceiling of r*L
    m = oracle.kept_count(L, w, r)
    assert m == min(L, max(min(w, L), exact))
    if exact >= min(w, L):
        assert m == exact
    if r == 1.0:
        assert m == L                           # Full CoT: nothing evicted


# ---------------------------------------------------------------- Eq. 2 score

def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


@pytest.mark.parametrize("L,G,w,D", [(1, 1, 1, 8), (3, 4, 1, 8), (17, 4, 4, 8), (64, 7, 4, 16),
                                     (257, 1, 32, 8), (40, 2, 40, 8), (10, 3, 16, 8)])
@pytest.mark.parametrize("causal", [True, False])
def test_score_mass_invariant(L, G, w, D, causal):
    """Every window row is a softmax that sums to one, so sum_j s_j = G * min(w, L)."""
    K = _rand((L, D), L)
    Q = _rand((G, w, D), L + 1)
    s = oracle.score_unit(K, Q, 1 / math.sqrt(D), causal)
    assert s.sum() == pytest.approx(G * min(w, L), rel=1e-12)
    assert (s >= 0).all()


def test_score_single_row_is_a_softmax():
    """G = w = 1: the window is the last token alone; causality does not bind
    (it sees every key), so s is one softmax row (scipy)."""
    K = _rand((50, 16), 1)
    q = _rand((1, 1, 16), 2)
    for causal in (True, False):
        s = oracle.score_unit(K, q, 0.25, causal)
        ref = scipy.special.softmax(0.25 * K @ q[0, 0])
        np.testing.assert_allclose(s, ref, rtol=1e-13, atol=0)


@pytest.mark.parametrize("L,w,G", [(20, 5, 3), (9, 9, 2), (33, 1, 4)])
def test_score_identical_keys_closed_form(L, w, G):
    """All keys equal: a causal window row at position p spreads mass 1/(p+1)
    over keys 0..p, so s_j = G * sum_{rows with p >= j} 1 / (p + 1)."""
    D = 8
    K = np.tile(_rand((1, D), 3), (L, 1))
    Q = _rand((G, w, D), 4)
    s = oracle.score_unit(K, Q, 0.3, True)
    pos = np.arange(L - w, L)
    ref = np.array([G * sum(1.0 / (p + 1) for p in pos if p >= j) for j in range(L)])
    np.testing.assert_allclose(s, ref, rtol=1e-12)
    s_nc = oracle.score_unit(K, Q, 0.3, False)
    np.testing.assert_allclose(s_nc, np.full(L, G * w / L), rtol=1e-12)


@pytest.mark.parametrize("L,G,w,D", [(37, 4, 8, 16), (64, 7, 16, 8), (5, 2, 5, 8)])
@pytest.mark.parametrize("causal", [True, False])
def test_score_equals_sdpa_with_identity_values(L, G, w, D, causal):
    """torch's scaled_dot_product_attention with V = identity returns the
    attention matrix itself; summing its rows over the window and the group
    gives Eq. 2 independently of the oracle's arithmetic."""
    K = _rand((L, D), 10 + L)
    Q = _rand((G, w, D), 11 + L)
    scale = 1 / math.sqrt(D)
    q = torch.from_numpy(Q)[None]                      # [1][G][w][D]
    k = torch.from_numpy(K)[None, None].expand(1, G, L, D)
    v = torch.eye(L, dtype=torch.float64)[None, None].expand(1, G, L, L)
    mask = None
    if causal:
        pos = torch.arange(L - w, L)
        mask = torch.arange(L)[None, :] <= pos[:, None]
    att = F.scaled_dot_product_attention(q, k, v, attn_mask=mask, scale=scale)
    ref = att.sum(dim=(0, 1, 2)).numpy()
    np.testing.assert_allclose(oracle.score_unit(K, Q, scale, causal), ref, rtol=1e-12, atol=1e-15)


def test_score_window_longer_than_cache():
    """w > L: window row t is the query of position L - w + t, so only the last
    L rows exist; they are the rows that see the whole (short) cache causally."""
    L, G, w, D = 6, 3, 10, 8
    K = _rand((L, D), 21)
    Q = _rand((G, w, D), 22)
    scale = 0.3
    q = torch.from_numpy(Q[:, w - L:])[None]
    k = torch.from_numpy(K)[None, None].expand(1, G, L, D)
    v = torch.eye(L, dtype=torch.float64)[None, None].expand(1, G, L, L)
    mask = torch.arange(L)[None, :] <= torch.arange(L)[:, None]
    ref = F.scaled_dot_product_attention(q, k, v, attn_mask=mask, scale=scale).sum(dim=(0, 1, 2)).numpy()
    np.testing.assert_allclose(oracle.score_unit(K, Q, scale, True), ref, rtol=1e-12)


def test_score_noncausal_permutation_equivariance():
    K = _rand((30, 8), 5)
    Q = _rand((3, 6, 8), 6)
    perm = np.random.default_rng(7).permutation(30)
    s = oracle.score_unit(K, Q, 0.4, False)
    sp = oracle.score_unit(K[perm], Q, 0.4, False)
    np.testing.assert_allclose(sp, s[perm], rtol=1e-13)


def test_score_zero_scale_is_uniform_causal_mass():
    """scale 0 makes every visible key equally likely: row p gives 1/(p+1) each."""
    L, w, G = 12, 4, 2
    K = _rand((L, 8), 8)
    Q = _rand((G, w, 8), 9)
    s = oracle.score_unit(K, Q, 0.0, True)
    ref = np.array([G * sum(1.0 / (p + 1) for p in range(L - w, L) if p >= j) for j in range(L)])
    np.testing.assert_allclose(s, ref, rtol=1e-13)


def test_score_cache_gqa_grouping():
    """Query head hq belongs to KV head hq // G: scoring a GQA cache equals
    scoring each KV head with its own slice of query heads."""
    NL, B, H, Cap, D, G, w = 2, 2, 3, 24, 8, 2, 4
    K = _rand((NL, B, H, Cap, D), 12)
    Q = _rand((NL, B, H * G, w, D), 13)
    lens = np.array([[[20, 24, 5], [24, 9, 17]]] * NL)
    s = oracle.score_cache(K, lens, Q, 0.35)
    for l in range(NL):
        for b in range(B):
            for h in range(H):
                L = lens[l, b, h]
                # brute force: loop over the group's query heads one at a time
                acc = np.zeros(L)
                for g in range(G):
                    acc += oracle.score_unit(K[l, b, h, :L], Q[l, b, h * G + g][None], 0.35)
                np.testing.assert_allclose(s[l, b, h, :L], acc, rtol=1e-13)
                assert (s[l, b, h, L:] == 0).all()


# ---------------------------------------------------------------- selection

def _valid_by_order(S, s, P):
    """A kept set is valid iff every kept prefix element outranks every evicted
    one under (score desc, position asc)."""
    kept = set(S)
    for a in kept:
        for b in range(P):
            if b in kept:
                continue
            if not (s[a] > s[b] or (s[a] == s[b] and a < b)):
                return False
    return True


@pytest.mark.parametrize("seed", range(12))
def test_select_matches_exhaustive_enumeration(seed):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(2, 11))
    w = int(rng.integers(1, L + 1))
    r = float(rng.choice([0.3, 0.45, 0.5, 0.75, 0.9, 1.0]))
    # small integer-valued scores produce plenty of ties
    s = rng.integers(0, 4, size=L).astype(np.float64) / 3.0
    idx = oracle.select_unit(s, L, w, r)
    w_eff = min(w, L)
    P = L - w_eff
    k = oracle.kept_count(L, w, r) - w_eff
    valid = [c for c in itertools.combinations(range(P), k) if _valid_by_order(c, s, P)]
    assert len(valid) == 1
    expect = list(valid[0]) + list(range(P, L))
    assert list(idx) == expect


@pytest.mark.parametrize("L,w,r", [(2048, 32, 0.62), (500, 64, 0.5), (70, 64, 0.3), (40, 64, 0.5)])
def test_select_invariants(L, w, r):
    s = np.abs(_rand(L, L))
    idx = oracle.select_unit(s, L, w, r)
    m = oracle.kept_count(L, w, r)
    w_eff = min(w, L)
    assert len(idx) == m
    assert (np.diff(idx) > 0).all()
    assert set(range(L - w_eff, L)) <= set(idx.tolist())
    kept_prefix = idx[idx < L - w_eff]
    evicted = np.setdiff1d(np.arange(L - w_eff), kept_prefix)
    if len(kept_prefix) and len(evicted):
        assert s[kept_prefix].min() >= s[evicted].max()


def test_select_special_cases():
    s = np.abs(_rand(100, 1))
    assert list(oracle.select_unit(s, 100, 8, 1.0)) == list(range(100))       # r = 1 keeps all
    eq = np.full(100, 0.5)
    k = oracle.kept_count(100, 8, 0.5) - 8
    assert list(oracle.select_unit(eq, 100, 8, 0.5)) == list(range(k)) + list(range(92, 100))


def test_compact_gathers_rows():
    K = np.arange(20)[:, None] * np.ones((1, 4))
    V = -K
    idx = np.array([0, 3, 4, 9, 19])
    k2, v2 = oracle.compact_unit(K, V, idx)
    assert (k2[:, 0] == idx).all() and (v2[:, 0] == -idx).all()


# ---------------------------------------------------------------- decode

@pytest.mark.parametrize("n,G,D", [(1, 1, 8), (5, 4, 16), (300, 7, 32), (77, 5, 8)])
def test_decode_equals_torch_sdpa_gqa(n, G, D):
    """Decode equals torch's SDPA (fp64, CPU) with GQA broadcasting."""
    H = 2
    K = _rand((H, n, D), n)
    V = _rand((H, n, D), n + 1)
    Q = _rand((H * G, D), n + 2)
    scale = 1 / math.sqrt(D)
    ref = F.scaled_dot_product_attention(torch.from_numpy(Q)[None, :, None, :], torch.from_numpy(K)[None],
                                         torch.from_numpy(V)[None], scale=scale, enable_gqa=True)[0, :, 0]
    for h in range(H):
        out, lse = oracle.decode_unit(K[h], V[h], n, Q[h * G:(h + 1) * G], scale)
        np.testing.assert_allclose(out, ref[h * G:(h + 1) * G].numpy(), rtol=1e-12, atol=1e-13)
        lref = scipy.special.logsumexp(scale * Q[h * G:(h + 1) * G] @ K[h].T, axis=1)
        np.testing.assert_allclose(lse, lref, rtol=1e-13)


def test_decode_special_cases():
    D = 16
    V = _rand((10, D), 1)
    K = _rand((10, D), 2)
    q = _rand((3, D), 3)
    out, _ = oracle.decode_unit(K, V, 1, q, 0.25)                     # one key: o = v0
    np.testing.assert_allclose(out, np.tile(V[0], (3, 1)), rtol=1e-14)
    Ks = np.tile(K[:1], (10, 1))                                      # identical keys: mean of V
    out, lse = oracle.decode_unit(Ks, V, 10, q, 0.25)
    np.testing.assert_allclose(out, np.tile(V.mean(axis=0), (3, 1)), rtol=1e-12)
    np.testing.assert_allclose(lse, 0.25 * q @ K[0] + math.log(10), rtol=1e-13)


def test_decode_append_equals_longer_cache():
    D = 8
    K = _rand((12, D), 4)
    V = _rand((12, D), 5)
    q = _rand((2, D), 6)
    a, la = oracle.decode_unit(K, V, 11, q, 0.3, K[11], V[11])
    b, lb = oracle.decode_unit(K, V, 12, q, 0.3)
    np.testing.assert_allclose(a, b, rtol=1e-14)
    np.testing.assert_allclose(la, lb, rtol=1e-14)


def test_decode_cache_appends_and_counts():
    NL, B, H, Cap, D, G = 1, 2, 2, 16, 8, 3
    K = _rand((NL, B, H, Cap, D), 7)
    V = _rand((NL, B, H, Cap, D), 8)
    lens = np.array([[[10, 4], [0, 15]]])
    Q = _rand((NL, B, H * G, D), 9)
    kn = _rand((NL, B, H, D), 10)
    vn = _rand((NL, B, H, D), 11)
    K0 = K.copy()
    out, lse = oracle.decode_cache(K, V, lens, Q, 0.2, kn, vn)
    assert (lens == np.array([[[11, 5], [1, 16]]])).all()
    np.testing.assert_array_equal(K[0, 0, 0, 10], kn[0, 0, 0])
    # a one-key cache (after append to an empty one) returns the appended value
    np.testing.assert_allclose(out[0, 1, 0:G], np.tile(vn[0, 1, 0], (G, 1)), rtol=1e-14)
    np.testing.assert_array_equal(K[0, 0, 1, :4], K0[0, 0, 1, :4])


# ---------------------------------------------------------------- Eq. 3 / Eq. 4

def test_penalty_bands_at_edges():
    lo, hi = np.float32(0.4), np.float32(0.8)
    b = (np.float32(0.0), np.float32(1.5), np.float32(3.0))          # paper form (0, beta/2, beta), beta = 3
    up = lambda x: np.nextafter(np.float32(x), np.float32(2))        # noqa: E731
    dn = lambda x: np.nextafter(np.float32(x), np.float32(-1))       # noqa: E731
    cases = [(0.0, 0.0), (dn(lo), 0.0), (lo, 0.0), (up(lo), 1.5), (0.6, 1.5), (dn(hi), 1.5),
             (hi, 3.0), (up(hi), 3.0), (1.0, 3.0)]
    for v, expect in cases:
        assert oracle.penalty_band(v, lo, hi, *b) == np.float32(expect), v


def test_penalty_touches_only_reflection_ids_exactly():
    rng = np.random.default_rng(3)
    z = (3 * rng.standard_normal((4, 1000))).astype(np.float32)
    R = [5, 17, 999, 17, 0]                                           # duplicate id 17
    v = np.array([0.1, 0.5, 0.9, 0.4], dtype=np.float32)
    out = oracle.logit_penalty(z, R, v, 0.4, 0.8, 0.0, 1.0, 3.0)
    beta = [0.0, 1.0, 3.0, 0.0]
    for b in range(4):
        for u in range(1000):
            if u in (0, 5, 17, 999):
                assert out[b, u] == np.float32(z[b, u] - np.float32(beta[b]))
            else:
                assert out[b, u].tobytes() == z[b, u].tobytes()


# ---------------------------------------------------------------- Eq. 5 / Eq. 6

def test_ppl_uniform_logits_equals_vocab():
    V = 977
    z = np.zeros((2, 5, V))
    x = np.zeros((2, 5), dtype=np.int64)
    ppl, stop = oracle.answer_ppl(z, x, 1.1)
    np.testing.assert_allclose(ppl, [V, V], rtol=1e-13)
    assert not stop.any()


def test_ppl_equals_exp_cross_entropy():
    rng = np.random.default_rng(4)
    z = 3 * rng.standard_normal((3, 7, 500))
    x = rng.integers(0, 500, size=(3, 7))
    ppl, _ = oracle.answer_ppl(z, x, 1.1)
    for b in range(3):
        ce = F.cross_entropy(torch.from_numpy(z[b]), torch.from_numpy(x[b]))
        assert ppl[b] == pytest.approx(math.exp(ce.item()), rel=1e-12)
    assert (ppl >= 1).all()


def test_ppl_confident_answer_stops():
    rng = np.random.default_rng(5)
    z = 3 * rng.standard_normal((2, 32, 2000))
    x = rng.integers(0, 2000, size=(2, 32))
    z[0, np.arange(32), x[0]] += 25.0                                 # sequence 0 is confident
    ppl, stop = oracle.answer_ppl(z, x, 1.1)
    assert ppl[0] < 1.1 and stop[0]
    assert ppl[1] > 1.1 and not stop[1]
