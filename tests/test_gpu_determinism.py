"""Repeatability: every kernel gives bitwise-identical results when called
again on the same inputs (fixed launch shapes and reduction orders, no
atomics in any reduction), and an invalid call changes nothing on the
device."""
import numpy as np
import pytest
import torch

from paper_2608_04771_amd import binding as B
from paper_2608_04771_amd import inputs as I

pytestmark = pytest.mark.gpu
REPEATS = 20


def _cache(seq_lens=(3000, 1777)):
    wl = I.WORKLOADS["7b16k"]
    ci = I.make_cache(wl, device=torch.device("cuda"), n_layers=3, seq_lens=list(seq_lens), capacity=3100)
    return wl, ci


def test_score_and_decode_repeat_bitwise():
    wl, ci = _cache()
    cache = B.KVCache(ci.k, ci.v, ci.length)
    s0 = B.reco_score(cache, ci.q_win, wl.window).clone()
    qs, _, _ = I.make_decode_inputs(wl, ci, 1, device=torch.device("cuda"))
    o0, l0 = (t.clone() for t in B.reco_decode_attn(cache, qs[0]))
    for _ in range(REPEATS):
        assert torch.equal(B.reco_score(cache, ci.q_win, wl.window), s0)
        o, l = B.reco_decode_attn(cache, qs[0])
        assert torch.equal(o, o0) and torch.equal(l, l0)
    assert torch.equal(cache.length, ci.length)


def test_select_compact_repeat_bitwise():
    wl, ci = _cache()
    cache0 = B.KVCache(ci.k, ci.v, ci.length)
    scores = B.reco_score(cache0, ci.q_win, wl.window)
    r = torch.tensor([0.55, 0.8], dtype=torch.float64, device="cuda")
    ref = None
    for _ in range(5):
        k, v, ln = ci.k.clone(), ci.v.clone(), ci.length.clone()
        c = B.KVCache(k, v, ln)
        kept = torch.full(scores.shape, -1, dtype=torch.int32, device="cuda")
        B.reco_select_compact(c, scores, r, wl.window, kept_idx=kept)
        torch.cuda.synchronize()
        got = (k, v, ln, kept)
        if ref is None:
            ref = got
        else:
            assert all(torch.equal(a, b) for a, b in zip(got, ref))


def test_penalty_sample_repeat_bitwise():
    z0 = I.make_logits(16, 152064, seed=3).cuda()
    ids = torch.from_numpy(I.make_reflection_ids(64, 152064, seed=4)).cuda()
    rew = torch.linspace(0, 1, 16, device="cuda")
    ref = None
    for _ in range(5):
        z = z0.clone()
        t = B.reco_penalty_sample(z, ids, rew, 0.4, 0.8, 0.0, 1.0, 3.0, 0.8, 123, 9)
        got = (z, t.clone())
        if ref is None:
            ref = got
        else:
            assert torch.equal(got[0], ref[0]) and torch.equal(got[1], ref[1])


def test_rejected_call_changes_nothing():
    wl, ci = _cache()
    cache = B.KVCache(ci.k, ci.v, ci.length)
    k0, l0 = ci.k.clone(), ci.length.clone()
    scores = torch.rand((3, 2, wl.n_kv_heads, 3100), device="cuda")
    r = torch.tensor([0.5, 0.5], dtype=torch.float64, device="cuda")
    tiny_ws = torch.empty(8, dtype=torch.uint8, device="cuda")
    with pytest.raises(RuntimeError, match="workspace"):
        B.reco_select_compact(cache, scores, r, wl.window, ws=tiny_ws)
    with pytest.raises(RuntimeError, match="workspace"):
        B.reco_decode_attn(cache, torch.zeros((3, 2, wl.n_q_heads, 128), dtype=torch.bfloat16, device="cuda"),
                           torch.zeros((3, 2, wl.n_kv_heads, 128), dtype=torch.bfloat16, device="cuda"),
                           torch.zeros((3, 2, wl.n_kv_heads, 128), dtype=torch.bfloat16, device="cuda"), ws=tiny_ws)
    torch.cuda.synchronize()
    assert torch.equal(ci.k, k0) and torch.equal(ci.length, l0)
