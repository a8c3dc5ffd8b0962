"""The 8B-shaped full trajectory at its real size, through the controller.

32 layers, 32 query / 8 KV heads, a 512-token prompt, 32,768 generated tokens
in reasoning steps of Geometric(mean 200) length, a Beta(2,5) process reward
and a compression at every step boundary, and the reflection penalty on a
128,256-token logit row per token.  The oracle checks sampled compressions
(scores, kept sets with ties excused, bit-exact gathered rows), sampled
decode outputs, sampled penalised rows and the final lengths; at every
compression the scores of every unit must sum to G * w (Eq. 2 conserves
each window row's probability mass)."""
import math
import time

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import (SCORE_RTOL, assert_decode_close, assert_lse_close, assert_mass_conserved,
                         assert_theta_precision, f64, kept_sets_match)
from paper_2608_04771_amd import inputs as I
from paper_2608_04771_amd import binding as B
from paper_2608_04771_amd.controller import RecoDecoder, RecoPolicy

pytestmark = pytest.mark.gpu


def test_8b_trajectory_full_size():
    wl = I.WORKLOADS["8b-trajectory"]
    dev = torch.device("cuda")
    ci = I.make_cache(wl, device=dev, capacity=8192)
    cache = B.KVCache(ci.k, ci.v, ci.length)
    NL, Bsz, H, Cap, D = cache.shape
    G, w, V = wl.group, wl.window, wl.vocab
    scale = 1.0 / math.sqrt(D)
    steps = I.make_step_lengths(wl.decode_steps, 200, wl.seed)
    rewards = I.make_rewards("beta25", len(steps), Bsz, wl.seed + 1)
    refl = I.make_reflection_ids(wl.n_reflection_ids, V, seed=wl.seed + 19)
    pol = RecoPolicy(retention="clamp", window=w, interval=0)
    dec = RecoDecoder(cache, wl.n_q_heads, pol, ci.q_win, torch.from_numpy(refl).to(dev), record_kept=True)

    units = [(0, 0, 0), (13, 0, 5), (31, 0, 7)]
    check_bounds = {5, len(steps) // 2, len(steps) - 2}
    check_tokens = {0, 4097, wl.decode_steps // 2 + 3, wl.decode_steps - 1}
    chunk = 1024
    tok = 0
    band = np.zeros(Bsz, dtype=np.float32)
    bounds = np.cumsum(steps)
    bi = 0
    checked = {"compress": 0, "decode": 0, "penalty": 0}
    worst_mass = 0.0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while tok < wl.decode_steps:
        n = min(chunk, wl.decode_steps - tok)
        qs, ks, vs = I.make_decode_inputs(wl, ci, n, seed_offset=tok, device=dev)
        z = I.make_logits(n * Bsz, V, seed=wl.seed + 100 + tok, device=dev).view(n, Bsz, V)
        for j in range(n):
            check_z = tok in check_tokens
            z0 = z[j].cpu().numpy().copy() if check_z else None
            out, lse = dec.decode(qs[j], ks[j], vs[j], logits=z[j])
            if check_z:
                torch.cuda.synchronize()
                for u in units:
                    l, b, h = u
                    m = int(cache.length[u].item())
                    ref, rl = oracle.decode_unit(f64(cache.k[u][:m]), f64(cache.v[u][:m]), m,
                                                 f64(qs[j][l, b, h * G:(h + 1) * G]), scale)
                    assert_decode_close(out[l, b, h * G:(h + 1) * G], ref, "bf16", f"token {tok} unit {u}")
                    assert_lse_close(lse[l, b, h * G:(h + 1) * G], rl, "bf16", f"token {tok} unit {u}")
                zr = oracle.logit_penalty(z0, refl, band, pol.tau_lo, pol.tau_hi, *pol.betas)
                assert z[j].cpu().numpy().tobytes() == zr.tobytes()
                checked["decode"] += 1
                checked["penalty"] += 1
            tok += 1
            if bi < len(bounds) and tok == bounds[bi]:
                check_c = bi in check_bounds
                if check_c:
                    torch.cuda.synchronize()
                    win = f64(dec.window_queries())
                    snap = {}
                    for u in units:
                        L = int(cache.length[u].item())
                        snap[u] = (L, f64(cache.k[u][:L]), f64(cache.v[u][:L]))
                L_before = dec.lengths()[0]
                dec.end_step([float(x) for x in rewards[bi]])
                band = rewards[bi].astype(np.float32)
                worst_mass = max(worst_mass, assert_mass_conserved(
                    dec.scores, torch.full((NL, Bsz, H), L_before, dtype=torch.int64), G, w,
                    f"8b step {bi}", verbose=False))
                if check_c:
                    torch.cuda.synchronize()
                    r = oracle.retention_from_reward(float(rewards[bi][0]))
                    for u in units:
                        l, b, h = u
                        L, K0, V0 = snap[u]
                        s_or = oracle.score_unit(K0, win[l, b, h * G:(h + 1) * G], scale)
                        s_gpu = dec.scores[u][:L].cpu().numpy().astype(np.float64)
                        assert (np.abs(s_gpu - s_or) / s_or).max() <= SCORE_RTOL
                        assert_theta_precision(s_gpu, s_or, L, w, r, f"8b step {bi} unit {u}")
                        kept = dec.kept[u].cpu().numpy()
                        ok, msg = kept_sets_match(kept, s_or, L, w, r)
                        assert ok, (bi, u, msg)
                        m = oracle.kept_count(L, w, r)
                        np.testing.assert_array_equal(f64(cache.k[u][:m]), K0[kept[:m]])
                        np.testing.assert_array_equal(f64(cache.v[u][:m]), V0[kept[:m]])
                    checked["compress"] += 1
                bi += 1
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    assert dec.dev_err.item() == 0
    lens = cache.length.cpu().numpy()
    assert (lens == dec.lengths()[0]).all()
    assert checked["compress"] == len(check_bounds) and checked["decode"] == len(check_tokens)
    print(f"8B trajectory: {wl.decode_steps} tokens, {len(steps)} compressions, final cache {lens.max()} rows, "
          f"{elapsed:.2f} s including input generation and checks; scores of every unit at every compression "
          f"sum to G*w within {worst_mass:.1e}")
