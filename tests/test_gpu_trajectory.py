"""GPU trajectory through the controller, replayed by the oracle event by event.

A prompt, then generated tokens in reasoning steps of geometric length; at each
step boundary a process reward (Beta(2,5)) drives the retention and the
penalty band.  Every decode output and lse, every reflection-penalised logit
row and every compression (kept sets, ties excused; lengths) is compared with
the oracle, which follows the GPU's selection after each compression so that
an excused tie cannot make the two trajectories diverge."""
import math

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import assert_decode_close, assert_lse_close, f64, kept_sets_match
from paper_2608_04771_amd import binding as B
from paper_2608_04771_amd import inputs as I
from paper_2608_04771_amd.controller import RecoDecoder, RecoPolicy

pytestmark = pytest.mark.gpu


VARIANTS = [
    ("clamp", "f32", {}), ("eq1", "f32", {}), ("clamp", "bf16", {}),
    ("eq1", "f32", {"delta": 0.0}),                                   # uniform retention: the paper's ablation
    ("clamp", "f32", {"layer_spread": 0.5}),                          # per-layer budgets
    ("eq1", "bf16", {"pool_kernel": 7, "pool_mode": "max"}),          # pooled scores
    ("clamp", "f32", {"pool_kernel": 5, "pool_mode": "mean", "layer_spread": 0.3}),
]


@pytest.mark.parametrize("retention,dtype,variant", VARIANTS)
def test_trajectory_matches_oracle_replay(retention, dtype, variant):
    NL, Bsz, H, Hq, D, w = 2, 2, 2, 8, 64, 16
    prompt, n_tokens, cap = 150, 360, 600
    vocab, n_refl = 1000, 16
    td = torch.float32 if dtype == "f32" else torch.bfloat16
    dev = torch.device("cuda")
    g = torch.Generator().manual_seed(77)
    rng = np.random.default_rng(77)
    k = torch.zeros((NL, Bsz, H, cap, D), dtype=td)
    v = torch.zeros_like(k)
    k[:, :, :, :prompt] = torch.randn((NL, Bsz, H, prompt, D), generator=g).to(td)
    v[:, :, :, :prompt] = torch.randn((NL, Bsz, H, prompt, D), generator=g).to(td)
    ln = torch.full((NL, Bsz, H), prompt, dtype=torch.int32)
    prompt_q = torch.randn((NL, Bsz, Hq, w, D), generator=g).to(td)
    qs = torch.randn((n_tokens, NL, Bsz, Hq, D), generator=g).to(td)
    ks = torch.randn((n_tokens, NL, Bsz, H, D), generator=g).to(td)
    vs = torch.randn((n_tokens, NL, Bsz, H, D), generator=g).to(td)
    logits = torch.randn((n_tokens, Bsz, vocab), generator=g) * 3
    refl = I.make_reflection_ids(n_refl, vocab, seed=5)
    # step boundaries: geometric step lengths, mean 30
    bounds, t = [], 0
    while True:
        t += int(rng.geometric(1 / 30))
        if t >= n_tokens:
            break
        bounds.append(t)
    rewards = rng.beta(2, 5, size=(len(bounds), Bsz))
    rewards[len(bounds) // 2] = 0.9                      # exercise the top band and the probe
    rewards[len(bounds) // 2 + 1] = 0.95

    pol = RecoPolicy(retention=retention, window=w, interval=0, **variant)
    cache = B.KVCache(k.to(dev), v.to(dev), ln.to(dev))
    dec = RecoDecoder(cache, Hq, pol, prompt_q.to(dev), torch.from_numpy(refl).to(dev), record_kept=True)

    K, V, lens = f64(k), f64(v), ln.numpy().astype(np.int64)
    win = f64(prompt_q)                                   # oracle window, chronological
    hist = [[] for _ in range(Bsz)]
    band = np.zeros(Bsz, dtype=np.float32)
    scale = 1 / math.sqrt(D)
    G = Hq // H
    z_dev = logits.to(dev)
    bi, probes, fed = 0, [], []
    for tok in range(n_tokens):
        q_dev = qs[tok].to(dev)
        if tok % 2:
            q_dev = dec.query_slot().copy_(q_dev)         # the caller writes the query into the ring itself
        out, lse = dec.decode(q_dev, ks[tok].to(dev), vs[tok].to(dev), logits=z_dev[tok])
        ref, rl = oracle.decode_cache(K, V, lens, f64(qs[tok]), scale, f64(ks[tok]), f64(vs[tok]))
        assert_decode_close(out, ref, dtype, f"token {tok}")
        assert_lse_close(lse, rl, dtype, f"token {tok}")
        zr = oracle.logit_penalty(logits[tok].numpy(), refl, band, 0.4, 0.8, 0.0, 1.0, 3.0)
        assert z_dev[tok].cpu().numpy().tobytes() == zr.tobytes(), f"penalty at token {tok}"
        win = np.concatenate([win[:, :, :, 1:], f64(qs[tok])[:, :, :, None]], axis=3)
        if bi < len(bounds) and tok + 1 == bounds[bi]:
            vb = rewards[bi]
            compressed, probe = dec.end_step(vb)
            probes.append(probe)
            fed.append(dec.last_score_stats_fed)
            if any(probe):
                # Answer probe (Eq. 5-6) on a synthetic 8-token answer; one
                # sequence's answer is made confident so both stop branches run.
                ans = torch.randn((Bsz, 8, vocab), generator=g) * 3
                ans_tok = torch.randint(0, vocab, (Bsz, 8), generator=g, dtype=torch.int32)
                ans[0, torch.arange(8), ans_tok[0].long()] += 25.0
                ppl, stop = dec.answer_ppl(ans.to(dev), ans_tok.to(dev))
                ppl_or, stop_or = oracle.answer_ppl(ans.numpy(), ans_tok.numpy(), pol.tau_p)
                np.testing.assert_allclose(ppl.cpu().numpy(), ppl_or, rtol=1e-5)
                assert (stop.cpu().numpy() == stop_or).all() and stop_or[0] and not stop_or[1]
            assert compressed
            r = []
            for b in range(Bsz):
                hist[b].append(float(vb[b]))
                r.append(oracle.retention_eq1(hist[b], 0.25, pol.delta) if retention == "eq1"
                         else oracle.retention_from_reward(vb[b]))
            s_or = oracle.score_cache(K, lens, win, scale)
            torch.cuda.synchronize()
            kept = dec.kept.cpu().numpy()
            for u in np.ndindex(NL, Bsz, H):
                L = int(lens[u])
                r_u = oracle.layer_retention(r[u[1]], u[0], NL, pol.layer_spread)
                s_u = s_or[u]
                if pol.pool_kernel > 1:
                    s_u = oracle.pool_scores(s_u, L, w, pol.pool_kernel, pol.pool_mode)
                ok, msg = kept_sets_match(kept[u], s_u, L, w, r_u)
                assert ok, (tok, u, msg)
                m = oracle.kept_count(L, w, r_u)
                idx = kept[u][:m]
                K[u][:m], V[u][:m] = K[u][idx].copy(), V[u][idx].copy()
                lens[u] = m
            assert (dec.cache.length.cpu().numpy() == lens).all()
            assert dec.layer_lengths() == [[int(lens[l, b, 0]) for l in range(NL)] for b in range(Bsz)]
            band = np.asarray(vb, dtype=np.float32)
            bi += 1
    assert dec.dev_err.item() == 0
    assert any(fed) and not all(fed)          # both the one-pass (decode statistics) and two-pass scoring ran
    expect = [[i > 0 and rewards[i][b] >= 0.8 and rewards[i - 1][b] >= 0.8 for b in range(Bsz)]
              for i in range(len(bounds))]
    assert probes == expect
    assert any(any(p) for p in probes)
    assert all(probes[len(bounds) // 2 + 1])
