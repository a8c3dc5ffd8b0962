"""Plant plausible mistakes in the CPU oracle and check that the pins catch them.

Each mutant replaces one oracle function by a copy with a single planted bug
(a dropped term, a wrong sign, index or comparison, a transposed reduction).
The test passes only if at least one pin of ``test_oracle_pins`` fails
against the mutant, i.e. the pins are strong enough to notice that bug."""
import math

import numpy as np
import pytest

import oracle
import oracle.reco_oracle as ro
import test_oracle_pins as pins
import test_oracle_policy as ppins
import test_oracle_sampling as spins

_ORIG_PPL = ro.answer_ppl
_ORIG_GUMBEL = ro.gumbel_noise
_ORIG_PENALTY = ro.logit_penalty
_ORIG_POOL = ro.pool_scores


# ----------------------------------------------------------------- mutants

def _score_generic(K, Qwin, scale, causal=True, *, use_scale=True, off_by_one=False, axis=1,
                   head_rows=False):
    K = np.asarray(K, dtype=np.float64)
    Qwin = np.asarray(Qwin, dtype=np.float64)
    L = K.shape[0]
    G, w, D = Qwin.shape
    w_eff = min(w, L)
    s = np.zeros(L)
    if L == 0:
        return s
    sel = Qwin[:, :w_eff, :] if head_rows else Qwin[:, w - w_eff:, :]
    rows = sel.reshape(G * w_eff, D)
    pos = np.tile(np.arange(L - w_eff, L), G)
    logits = (scale if use_scale else 1.0) * (rows @ K.T)
    if causal:
        vis = (np.arange(L)[None, :] < pos[:, None]) if off_by_one else (np.arange(L)[None, :] <= pos[:, None])
        vis[:, 0] = True
        logits = np.where(vis, logits, -np.inf)
    logits = logits - logits.max(axis=1, keepdims=True)
    e = np.exp(logits)
    if axis == 1:
        p = e / e.sum(axis=1, keepdims=True)
    else:
        p = e / e.sum(axis=0, keepdims=True)
        p = np.nan_to_num(p)
    return s + p.sum(axis=0)


SCORE_MUTANTS = {
    "dropped_scale": lambda K, Q, sc, c=True: _score_generic(K, Q, sc, c, use_scale=False),
    "always_noncausal": lambda K, Q, sc, c=True: _score_generic(K, Q, sc, False),
    "causal_off_by_one": lambda K, Q, sc, c=True: _score_generic(K, Q, sc, c, off_by_one=True),
    "softmax_over_queries": lambda K, Q, sc, c=True: _score_generic(K, Q, sc, c, axis=0),
    "window_rows_from_the_front": lambda K, Q, sc, c=True: _score_generic(K, Q, sc, c, head_rows=True),
}

SCORE_PINS = [
    lambda: pins.test_score_mass_invariant(17, 4, 4, 8, True),
    lambda: pins.test_score_mass_invariant(40, 2, 40, 8, False),
    pins.test_score_single_row_is_a_softmax,
    lambda: pins.test_score_identical_keys_closed_form(20, 5, 3),
    lambda: pins.test_score_equals_sdpa_with_identity_values(37, 4, 8, 16, True),
    lambda: pins.test_score_equals_sdpa_with_identity_values(37, 4, 8, 16, False),
    lambda: pins.test_score_equals_sdpa_with_identity_values(5, 2, 5, 8, True),
    pins.test_score_zero_scale_is_uniform_causal_mass,
    pins.test_score_window_longer_than_cache,
]


def _select_generic(s, L, w, r, *, desc=True, later_first=False, force_window=True):
    L = int(L)
    w_eff = min(int(w), L)
    m = ro.kept_count(L, w, r)
    if not force_window:
        order = np.lexsort((np.arange(L), -np.asarray(s)[:L]))
        return np.sort(order[:m])
    k = m - w_eff
    P = L - w_eff
    prefix = np.asarray(s, dtype=np.float64)[:P]
    pos_key = -np.arange(P) if later_first else np.arange(P)
    order = np.lexsort((pos_key, -prefix if desc else prefix))
    return np.concatenate([np.sort(order[:k]), np.arange(P, L)])


SELECT_MUTANTS = {
    "keeps_lowest_scores": lambda s, L, w, r: _select_generic(s, L, w, r, desc=False),
    "ties_to_later_position": lambda s, L, w, r: _select_generic(s, L, w, r, later_first=True),
    "window_not_forced": lambda s, L, w, r: _select_generic(s, L, w, r, force_window=False),
}

SELECT_PINS = [lambda seed=seed: pins.test_select_matches_exhaustive_enumeration(seed) for seed in range(12)] + [
    lambda: pins.test_select_invariants(500, 64, 0.5),
    pins.test_select_special_cases,
]


def _kept_floor(L, w, r):
    w_eff = min(int(w), int(L))
    return min(int(L), max(w_eff, math.floor(float(r) * float(L))))


def _kept_window_outside(L, w, r):
    w_eff = min(int(w), int(L))
    return min(int(L), w_eff + math.ceil(float(r) * float(L)))


BUDGET_MUTANTS = {"floor_instead_of_ceil": _kept_floor, "window_outside_budget": _kept_window_outside}
BUDGET_PINS = [lambda a=a: pins.test_kept_count_is_exact_ceiling(*a)
               for a in [(2048, 32, 0.75), (1001, 32, 0.75), (16383, 64, 0.6), (7, 32, 0.5), (100, 1, 1.0)]]


def _decode_generic(K, V, n, Q, scale, k_new=None, v_new=None, *, use_scale=True, append=True,
                    lse_drop_logz=False):
    K = np.asarray(K, dtype=np.float64)[:n]
    V = np.asarray(V, dtype=np.float64)[:n]
    if k_new is not None and append:
        K = np.vstack([K, np.asarray(k_new)[None, :]])
        V = np.vstack([V, np.asarray(v_new)[None, :]])
    if K.shape[0] == 0:
        return np.zeros((Q.shape[0], Q.shape[1])), np.full(Q.shape[0], -np.inf)
    a = (scale if use_scale else 1.0) * (np.asarray(Q) @ K.T)
    M = a.max(axis=1, keepdims=True)
    e = np.exp(a - M)
    Z = e.sum(axis=1, keepdims=True)
    lse = M[:, 0] if lse_drop_logz else (M + np.log(Z))[:, 0]
    return (e @ V) / Z, lse


DECODE_MUTANTS = {
    "dropped_scale": lambda *a: _decode_generic(*a, use_scale=False),
    "attends_before_append": lambda *a: _decode_generic(*a, append=False),
    "lse_without_log_z": lambda *a: _decode_generic(*a, lse_drop_logz=True),
}
DECODE_PINS = [lambda: pins.test_decode_equals_torch_sdpa_gqa(300, 7, 32), pins.test_decode_special_cases,
               pins.test_decode_append_equals_longer_cache, pins.test_decode_cache_appends_and_counts]


def _decode_cache_wrong_group(K, V, lens, Q, scale, k_new=None, v_new=None, units=None):
    NL, B, H, Cap, D = K.shape
    Hq = Q.shape[2]
    G = Hq // H
    out = np.zeros((NL, B, Hq, D))
    lse = np.zeros((NL, B, Hq))
    for l in range(NL):
        for b in range(B):
            for h in range(H):
                n = int(lens[l, b, h])
                heads = list(range(h, Hq, H))            # planted: hq % H instead of hq // G
                o, z = ro.decode_unit(K[l, b, h], V[l, b, h], n, Q[l, b, heads], scale,
                                      None if k_new is None else k_new[l, b, h],
                                      None if v_new is None else v_new[l, b, h])
                out[l, b, heads] = o
                lse[l, b, heads] = z
                if k_new is not None:
                    K[l, b, h, n] = k_new[l, b, h]
                    V[l, b, h, n] = v_new[l, b, h]
                    lens[l, b, h] = n + 1
    return out, lse


def _pin_decode_cache_vs_sdpa():
    """Cache-level decode vs torch SDPA with GQA (query head hq -> kv head hq // G)."""
    import torch
    import torch.nn.functional as F
    NL, B, H, Cap, D, G = 1, 1, 2, 9, 8, 3
    rng = np.random.default_rng(1)
    K = rng.standard_normal((NL, B, H, Cap, D))
    V = rng.standard_normal((NL, B, H, Cap, D))
    Q = rng.standard_normal((NL, B, H * G, D))
    lens = np.full((NL, B, H), Cap)
    out, _ = oracle.decode_cache(K.copy(), V.copy(), lens.copy(), Q, 0.3)
    ref = F.scaled_dot_product_attention(torch.from_numpy(Q[0, 0])[None, :, None], torch.from_numpy(K[0, 0])[None],
                                         torch.from_numpy(V[0, 0])[None], scale=0.3, enable_gqa=True)[0, :, 0]
    np.testing.assert_allclose(out[0, 0], ref.numpy(), rtol=1e-12)


def _penalty_strict_low(z, refl_ids, reward, tau_lo, tau_hi, b_lo, b_mid, b_hi):
    out = np.array(z, dtype=np.float32, copy=True)
    for b in range(out.shape[0]):
        v = np.float32(reward[b])
        beta = b_lo if v < np.float32(tau_lo) else (b_hi if v >= np.float32(tau_hi) else b_mid)
        for u in set(int(x) for x in refl_ids):
            out[b, u] = np.float32(out[b, u] - np.float32(beta))
    return out


def _penalty_dupes(z, refl_ids, reward, tau_lo, tau_hi, b_lo, b_mid, b_hi):
    out = np.array(z, dtype=np.float32, copy=True)
    for b in range(out.shape[0]):
        beta = ro.penalty_band(reward[b], tau_lo, tau_hi, b_lo, b_mid, b_hi)
        for u in refl_ids:                                  # planted: duplicates penalised twice
            out[b, u] = np.float32(out[b, u] - beta)
    return out


def _band_strict_low(v, tau_lo, tau_hi, b_lo, b_mid, b_hi):
    v = np.float32(v)
    if v < np.float32(tau_lo):
        return np.float32(b_lo)
    if v >= np.float32(tau_hi):
        return np.float32(b_hi)
    return np.float32(b_mid)


def _ppl_log2(logits, tokens, tau_p):
    ppl, _ = _ORIG_PPL(logits, tokens, tau_p)
    ppl = np.exp(np.log(ppl) / math.log(2))
    return ppl, ppl <= tau_p


def _ppl_sum(logits, tokens, tau_p):
    ppl, _ = _ORIG_PPL(logits, tokens, tau_p)
    n = np.asarray(tokens).shape[1]
    ppl = ppl ** n
    return ppl, ppl <= tau_p


def _gumbel_sign_flipped(row, vocab, seed, offset):
    return (-_ORIG_GUMBEL(row, vocab, seed, offset)).astype(np.float32)


def _uniform_missing_half_cell(x):
    # planted: U = k * 2^-23 without the half-cell offset, so U can be 0 and is biased low
    k = (np.asarray(x, dtype=np.uint32) >> np.uint32(9)).astype(np.float32)
    return (k * np.float32(2.0 ** -23)).astype(np.float32)


def _uniform_24_bits(x):
    # planted: a 24-bit grid, whose top midpoint 1 - 2^-25 rounds to 1.0 in float32
    k = (np.asarray(x, dtype=np.uint32) >> np.uint32(8)).astype(np.float32)
    return (k * np.float32(2.0 ** -24) + np.float32(2.0 ** -25)).astype(np.float32)


def _sample_without_penalty(z, refl_ids, reward, tau_lo, tau_hi, b_lo, b_mid, b_hi, temperature, seed, offset):
    zp = np.array(z, dtype=np.float32, copy=True)            # planted: penalty never applied
    vals = zp if temperature == 0 else np.stack([zp[b] / np.float32(temperature) + _ORIG_GUMBEL(b, zp.shape[1], seed, offset)
                                                 for b in range(zp.shape[0])])
    return zp, np.argmax(vals, axis=1), vals


def _sample_temperature_multiplied(z, refl_ids, reward, tau_lo, tau_hi, b_lo, b_mid, b_hi, temperature, seed, offset):
    zp = _ORIG_PENALTY(z, refl_ids, reward, tau_lo, tau_hi, b_lo, b_mid, b_hi)
    vals = zp if temperature == 0 else np.stack([zp[b] * np.float32(temperature) + _ORIG_GUMBEL(b, zp.shape[1], seed, offset)
                                                 for b in range(zp.shape[0])])
    return zp, np.argmax(vals, axis=1), vals


def _layer_ret_ascending(r, layer, n_layers, spread):
    # planted: the slope runs the wrong way (more cache at the top layers)
    t = 0.0 if n_layers == 1 else layer / (n_layers - 1)
    return min(1.0, r * (1.0 - spread * (1.0 - 2.0 * t)))


def _layer_ret_uncapped(r, layer, n_layers, spread):
    t = 0.0 if n_layers == 1 else layer / (n_layers - 1)
    return r * (1.0 + spread * (1.0 - 2.0 * t))                       # planted: no cap at 1


def _layer_ret_half_slope(r, layer, n_layers, spread):
    t = 0.0 if n_layers == 1 else layer / (n_layers - 1)
    return min(1.0, r * (1.0 + spread * (1.0 - t)))                   # planted: mean is not r


def _pool_including_window(s, L, w, kernel, mode):
    # planted: the window positions take part in the pooling
    return _ORIG_POOL(s, L, 0, kernel, mode)[:L] if L else np.zeros(0)


def _pool_wide(s, L, w, kernel, mode):
    return _ORIG_POOL(s, L, w, kernel + 2, mode)                     # planted: half width off by one


def _pool_mean_over_kernel(s, L, w, kernel, mode):
    # planted: the mean divides by the kernel size even where the window is cut at the edges
    out = _ORIG_POOL(s, L, w, kernel, mode)
    if mode != "mean":
        return out
    P = L - min(w, L)
    h = kernel // 2
    for j in range(P):
        cnt = min(P, j + h + 1) - max(0, j - h)
        out[j] = out[j] * cnt / kernel
    return out


def _pool_shifted(s, L, w, kernel, mode):
    # planted: the pooling window is not centred (covers j .. j + kernel - 1)
    s = np.asarray(s, dtype=np.float64)
    out = s[:L].copy()
    P = L - min(w, L)
    for j in range(P):
        seg = s[j:min(P, j + kernel)]
        out[j] = seg.max() if mode == "max" else seg.mean()
    return out


LAYER_PINS = [ppins.test_layer_retention_is_a_descending_line_with_mean_r, ppins.test_layer_retention_cap_and_edges,
              ppins.test_compress_cache_takes_per_layer_retention]
POOL_PINS = [ppins.test_pool_kernel_one_is_identity_and_constant_stays_constant,
             ppins.test_pool_max_spreads_a_spike_over_the_kernel_width, ppins.test_pool_mean_of_a_ramp_is_the_ramp_inside,
             ppins.test_pool_leaves_the_window_alone_and_ignores_it]

SAMPLING_PINS = [spins.test_gumbel_noise_moments, spins.test_greedy_is_argmax_of_penalised_logits,
                 spins.test_sampling_distribution_is_softmax_of_penalised_logits]

CASES = (
    [("score_unit", name, fn, SCORE_PINS) for name, fn in SCORE_MUTANTS.items()]
    + [("select_unit", name, fn, SELECT_PINS) for name, fn in SELECT_MUTANTS.items()]
    + [("kept_count", name, fn, BUDGET_PINS) for name, fn in BUDGET_MUTANTS.items()]
    + [("decode_unit", name, fn, DECODE_PINS) for name, fn in DECODE_MUTANTS.items()]
    + [("decode_cache", "gqa_modulo_mapping", _decode_cache_wrong_group, [_pin_decode_cache_vs_sdpa])]
    + [("logit_penalty", "strict_low_band", _penalty_strict_low, [pins.test_penalty_touches_only_reflection_ids_exactly]),
       ("penalty_band", "strict_low_band", _band_strict_low, [pins.test_penalty_bands_at_edges]),
       ("logit_penalty", "duplicates_twice", _penalty_dupes, [pins.test_penalty_touches_only_reflection_ids_exactly]),
       ("answer_ppl", "log_base_two", _ppl_log2, [pins.test_ppl_uniform_logits_equals_vocab,
                                                  pins.test_ppl_equals_exp_cross_entropy]),
       ("answer_ppl", "sum_not_mean", _ppl_sum, [pins.test_ppl_uniform_logits_equals_vocab,
                                                 pins.test_ppl_equals_exp_cross_entropy]),
       ("gumbel_noise", "sign_flipped", _gumbel_sign_flipped, SAMPLING_PINS),
       ("uniform_from_bits", "missing_half_cell", _uniform_missing_half_cell,
        [spins.test_uniform_grid_is_open_and_symmetric]),
       ("uniform_from_bits", "grid_of_24_bits", _uniform_24_bits, [spins.test_uniform_grid_is_open_and_symmetric]),
       ("penalty_sample", "penalty_skipped", _sample_without_penalty, SAMPLING_PINS),
       ("penalty_sample", "temperature_multiplied", _sample_temperature_multiplied, SAMPLING_PINS),
       ("layer_retention", "ascending", _layer_ret_ascending, LAYER_PINS),
       ("layer_retention", "uncapped", _layer_ret_uncapped, LAYER_PINS),
       ("layer_retention", "half_slope", _layer_ret_half_slope, LAYER_PINS),
       ("pool_scores", "includes_window", _pool_including_window, POOL_PINS),
       ("pool_scores", "too_wide", _pool_wide, POOL_PINS),
       ("pool_scores", "mean_over_kernel_size", _pool_mean_over_kernel, POOL_PINS),
       ("pool_scores", "not_centred", _pool_shifted, POOL_PINS)]
)


def test_unmutated_oracle_passes_the_pins_used_here():
    for pin in (_pin_decode_cache_vs_sdpa,):
        pin()


@pytest.mark.parametrize("target,name,fn,pin_list", CASES, ids=[f"{c[0]}-{c[1]}" for c in CASES])
def test_pins_catch_planted_mistake(monkeypatch, target, name, fn, pin_list):
    monkeypatch.setattr(ro, target, fn)
    monkeypatch.setattr(oracle, target, fn, raising=False)
    caught = 0
    for pin in pin_list:
        try:
            pin()
        except (AssertionError, ValueError, IndexError):
            caught += 1
    assert caught > 0, f"no pin noticed mutant {target}:{name}"
