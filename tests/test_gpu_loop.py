"""End-to-end GPU parity of the hot path: score -> select/compact -> decode
steps, on the tiny workload in full and on the 7B-shaped 16K workload at its
full size in the launch configuration the bench times (all layers per call),
checked on sampled units and steps."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import (SCORE_RTOL, assert_decode_close, assert_lse_close, assert_theta_precision, f64,
                         kept_sets_match, upload)
from paper_2608_04771_amd import binding as B
from paper_2608_04771_amd import inputs as I

pytestmark = pytest.mark.gpu


def _compress_gpu(wl, ci, cache):
    r = np.array([B.reco_retention_from_reward(float(v)) for v in ci.reward], dtype=np.float64)
    scores = B.reco_score(cache, ci.q_win.cuda(), wl.window)
    kept = torch.full(tuple(cache.shape[:4]), -1, dtype=torch.int32, device="cuda")
    dev_err = torch.zeros(1, dtype=torch.int32, device="cuda")
    B.reco_select_compact(cache, scores, torch.from_numpy(r).cuda(), wl.window, kept_idx=kept, dev_err=dev_err)
    torch.cuda.synchronize()
    assert dev_err.item() == 0
    return r, scores.cpu().numpy(), kept.cpu().numpy()


def test_tiny_workload_full_loop():
    wl = I.WORKLOADS["tiny"]
    ci = I.make_cache(wl)
    cache = upload(ci)
    K0, V0 = f64(ci.k), f64(ci.v)
    r, s_gpu, kept = _compress_gpu(wl, ci, cache)
    s_or = oracle.score_cache(K0, ci.length.numpy(), f64(ci.q_win), 1 / np.sqrt(wl.head_dim))
    # the oracle's own compression
    _, idx_or, K, V, lens = oracle.compress_cache(K0, V0, ci.length.numpy().astype(np.int64), f64(ci.q_win), r,
                                                  wl.window, 1 / np.sqrt(wl.head_dim))
    exact = True
    for h in range(wl.n_kv_heads):
        L = int(ci.seq_len[0])
        ok, msg = kept_sets_match(kept[0, 0, h], s_or[0, 0, h], L, wl.window, r[0])
        assert ok, msg
        assert_theta_precision(s_gpu[0, 0, h], s_or[0, 0, h], L, wl.window, r[0], f"tiny loop head {h}")
        exact = exact and msg == "exact"
        m = len(idx_or[(0, 0, h)])
        if msg != "exact":
            # continue from the GPU's (equally valid) selection
            K[0, 0, h, :m] = K0[0, 0, h][kept[0, 0, h, :m]]
            V[0, 0, h, :m] = V0[0, 0, h][kept[0, 0, h, :m]]
    assert (cache.length.cpu().numpy() == lens).all()
    assert np.array_equal(f64(cache.k)[..., :int(lens.max()), :], K[..., :int(lens.max()), :])
    qs, ks, vs = I.make_decode_inputs(wl, ci, wl.decode_steps)
    for s in range(wl.decode_steps):
        out, lse = B.reco_decode_attn(cache, qs[s].cuda(), ks[s].cuda(), vs[s].cuda())
        ref, rl = oracle.decode_cache(K, V, lens, f64(qs[s]), 1 / np.sqrt(wl.head_dim), f64(ks[s]), f64(vs[s]))
        assert_decode_close(out, ref, "f32", f"step {s}")
        assert_lse_close(lse, rl, "f32", f"step {s}")
    print("tiny loop: selection", "exact" if exact else "with excused ties")


def test_7b16k_full_size_sampled():
    """28 layers x 4 KV heads, 16,384 cached tokens, bf16: every call covers all
    layers (the bench's launch configuration).  Sampled units are checked
    against the oracle for scores, kept sets, gathered rows and decode steps;
    all units are checked for lengths and finiteness."""
    wl = I.WORKLOADS["7b16k"]
    ci = I.make_cache(wl)
    cache = upload(ci)
    k_before = cache.k.clone()
    r, s_gpu, kept = _compress_gpu(wl, ci, cache)
    L = int(ci.seq_len[0])
    m = oracle.kept_count(L, wl.window, float(r[0]))
    assert (cache.length.cpu().numpy() == m).all()
    G = wl.group
    scale = 1 / np.sqrt(wl.head_dim)
    units = [(0, 0, 0), (5, 0, 3), (13, 0, 1), (27, 0, 2)]
    for (l, b, h) in units:
        Kf = f64(ci.k[l, b, h, :L])
        s_or = oracle.score_unit(Kf, f64(ci.q_win[l, b, h * G:(h + 1) * G]), scale)
        rel = np.abs(s_gpu[l, b, h, :L] - s_or) / s_or
        assert rel.max() <= SCORE_RTOL, rel.max()
        assert_theta_precision(s_gpu[l, b, h], s_or, L, wl.window, float(r[0]), f"7b unit {(l, b, h)}")
        ok, msg = kept_sets_match(kept[l, b, h], s_or, L, wl.window, float(r[0]))
        assert ok, msg
        idx = torch.from_numpy(kept[l, b, h, :m].astype(np.int64)).cuda()
        assert torch.equal(cache.k[l, b, h, :m], k_before[l, b, h][idx])
    # gathered rows of every unit are bit-exact copies
    kk = torch.from_numpy(kept[..., :m].astype(np.int64)).cuda()
    gathered = torch.gather(k_before, 3, kk[..., None].expand(-1, -1, -1, -1, wl.head_dim))
    assert torch.equal(cache.k[:, :, :, :m], gathered)
    del gathered, k_before
    steps = wl.decode_steps
    qs, ks, vs = I.make_decode_inputs(wl, ci, steps)
    check_steps = {0, steps // 2, steps - 1}
    ws = B.decode_workspace(cache, wl.n_q_heads)
    w = wl.window
    stats = torch.empty((steps, wl.n_layers, 1, wl.n_q_heads, 2), dtype=torch.float32, device="cuda")
    for s in range(steps):
        out, lse = B.reco_decode_attn(cache, qs[s].cuda(), ks[s].cuda(), vs[s].cuda(), ws=ws, row_stats=stats[s])
        if s in check_steps:
            torch.cuda.synchronize()
            assert torch.isfinite(out.float()).all()
            for (l, b, h) in units:
                n = m + s + 1                       # the call appended row m + s
                Kc = f64(cache.k[l, b, h, :n])
                Vc = f64(cache.v[l, b, h, :n])
                ref, rl = oracle.decode_unit(Kc, Vc, n, f64(qs[s][l, b, h * G:(h + 1) * G]), scale)
                assert_decode_close(out[l, b, h * G:(h + 1) * G], ref, "bf16", f"step {s} unit {(l, b, h)}")
                assert_lse_close(lse[l, b, h * G:(h + 1) * G], rl, "bf16", f"step {s} unit {(l, b, h)}")
    assert (cache.length.cpu().numpy() == m + steps).all()
    # One-pass scoring of the post-decode cache, fed with the decode statistics
    # of the last w tokens (no compression since), against the two-pass kernels
    # and the oracle on the sampled units.
    q_win = torch.stack([q.cuda() for q in qs[-w:]], dim=3).contiguous()        # [NL][B][Hq][w][D]
    st_win = stats[-w:].permute(1, 2, 3, 0, 4).contiguous()
    s_fed = B.reco_score(cache, q_win, w, row_stats=st_win).cpu().numpy().astype(np.float64)
    s_two = B.reco_score(cache, q_win, w).cpu().numpy().astype(np.float64)
    n = m + steps
    big = s_two[..., :n] > 1e-20
    assert (np.abs(s_fed[..., :n] - s_two[..., :n])[big] / s_two[..., :n][big]).max() <= SCORE_RTOL
    for (l, b, h) in units:
        s_or = oracle.score_unit(f64(cache.k[l, b, h, :n]), f64(q_win[l, b, h * G:(h + 1) * G]), scale)
        assert (np.abs(s_fed[l, b, h, :n] - s_or) / s_or).max() <= SCORE_RTOL
        assert_theta_precision(s_fed[l, b, h], s_or, n, w, 0.5, f"7b one-pass unit {(l, b, h)}")
        ok, msg = kept_sets_match(oracle.select_unit(s_fed[l, b, h], n, w, 0.5), s_or, n, w, 0.5)
        assert ok, msg
