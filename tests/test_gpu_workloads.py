"""Full-size parity of the ragged 7B batch and the 32B-shaped 64K workloads.

The caches are drawn on the GPU with a seeded generator (tens to a hundred GB
do not fit the host path), every call covers all layers, and the oracle checks
sampled units by reading them back: scores, kept sets (ties excused),
bit-exact gathered rows, decode outputs and lse; lengths and the mass
conservation of the scores (each unit's scores sum to G * min(w, L)) are
checked for every unit, and the decode outputs and lse of every unit
against a plain PyTorch fp32 attention on the device.  The 32B test also
runs the reflection penalty and the answer perplexity on its logit shapes."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import (SCORE_RTOL, assert_decode_all_units, assert_decode_close, assert_lse_close,
                         assert_mass_conserved, assert_theta_precision, f64, kept_sets_match)
from paper_2608_04771_amd import binding as B
from paper_2608_04771_amd import inputs as I

pytestmark = pytest.mark.gpu


def _run_workload(wl, units, decode_steps, check_steps, seq_lens=None):
    dev = torch.device("cuda")
    ci = I.make_cache(wl, device=dev, seq_lens=seq_lens)
    cache = B.KVCache(ci.k, ci.v, ci.length)
    NL, Bsz, H, Cap, D = cache.shape
    assert (NL, H, D) == (wl.n_layers, wl.n_kv_heads, wl.head_dim) and Bsz == wl.batch
    G = wl.group
    scale = 1.0 / np.sqrt(D)
    r = np.array([oracle.retention_from_reward(float(v)) for v in ci.reward])
    lens0 = ci.length.cpu().numpy()
    before = {u: (f64(ci.k[u][:int(lens0[u])]), f64(ci.v[u][:int(lens0[u])])) for u in units}
    qwin = {u: f64(ci.q_win[u[0], u[1], u[2] * G:(u[2] + 1) * G]) for u in units}

    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    ev[0].record()
    scores = B.reco_score(cache, ci.q_win, wl.window)
    kept = torch.full((NL, Bsz, H, Cap), -1, dtype=torch.int32, device=dev)
    dev_err = torch.zeros(1, dtype=torch.int32, device=dev)
    ev[1].record()
    B.reco_select_compact(cache, scores, torch.from_numpy(r).to(dev), wl.window, kept_idx=kept, dev_err=dev_err)
    ev[2].record()
    torch.cuda.synchronize()
    print(f"{wl.name}: score {ev[0].elapsed_time(ev[1]):.2f} ms, select+compact {ev[1].elapsed_time(ev[2]):.2f} ms "
          f"over {int(lens0.sum())} cached rows")
    assert dev_err.item() == 0
    assert_mass_conserved(scores, torch.from_numpy(lens0.astype(np.int64)), G, wl.window, wl.name)
    m_all = np.array([[oracle.kept_count(int(lens0[0, b, 0]), wl.window, r[b]) for b in range(Bsz)]])
    lens1 = cache.length.cpu().numpy()
    assert (lens1 == m_all[:, :, None]).all()

    for u in units:
        L = int(lens0[u])
        K0, V0 = before[u]
        s_or = oracle.score_unit(K0, qwin[u], scale)
        s_gpu = scores[u][:L].cpu().numpy().astype(np.float64)
        rel = np.abs(s_gpu - s_or) / s_or
        assert rel.max() <= SCORE_RTOL, (u, rel.max())
        assert_theta_precision(s_gpu, s_or, L, wl.window, r[u[1]], f"{wl.name} unit {u}")
        ok, msg = kept_sets_match(kept[u].cpu().numpy(), s_or, L, wl.window, r[u[1]])
        assert ok, (u, msg)
        m = int(lens1[u])
        idx = kept[u][:m].cpu().numpy()
        np.testing.assert_array_equal(f64(cache.k[u][:m]), K0[idx])
        np.testing.assert_array_equal(f64(cache.v[u][:m]), V0[idx])

    qs, ks, vs = I.make_decode_inputs(wl, ci, decode_steps, device=dev)
    for s in range(decode_steps):
        out, lse = B.reco_decode_attn(cache, qs[s], ks[s], vs[s], dev_err=dev_err)
        if s in check_steps:
            torch.cuda.synchronize()
            assert torch.isfinite(out.float()).all()
            assert_decode_all_units(cache, qs[s], out, lse, torch.from_numpy(lens1.astype(np.int64)) + s + 1,
                                    scale, f"{wl.name} step {s}")
            for u in units:
                n = int(lens1[u]) + s + 1
                l, b, h = u
                ref, rl = oracle.decode_unit(f64(cache.k[u][:n]), f64(cache.v[u][:n]), n,
                                             f64(qs[s][l, b, h * G:(h + 1) * G]), scale)
                assert_decode_close(out[l, b, h * G:(h + 1) * G], ref, "bf16", f"step {s} unit {u}")
                assert_lse_close(lse[l, b, h * G:(h + 1) * G], rl, "bf16", f"step {s} unit {u}")
    torch.cuda.synchronize()
    assert dev_err.item() == 0
    assert (cache.length.cpu().numpy() == lens1 + decode_steps).all()
    # Timing of back-to-back decode calls (all layers per call) after the checks.
    n_rows = int(cache.length.sum().item())
    ws = B.decode_workspace(cache, wl.n_q_heads)
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for s in range(2):
        B.reco_decode_attn(cache, qs[s], ks[s], vs[s], ws=ws)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / 2
    gb = (n_rows + 1.5 * cache.length.numel()) * 2 * D * 2 / 1e9
    print(f"{wl.name}: decode call {ms:.2f} ms for {gb:.1f} GB of K/V -> {gb / ms:.2f} TB/s")
    return ci, cache


def test_7b_ragged_batch32_full_size():
    """32 sequences with lengths ~ U[4096, 32768] and per-sequence rewards:
    ragged per-unit lengths after compression, one workgroup per unit."""
    wl = I.WORKLOADS["7b-batch32"]
    units = [(0, 0, 0), (3, 7, 2), (11, 13, 1), (20, 21, 3), (27, 31, 0)]
    _run_workload(wl, units, decode_steps=6, check_steps={0, 5})


def test_32b_64k_full_size():
    """64 layers x 8 sequences x 8 KV heads at 65,536 cached tokens (GQA 5),
    window 32; plus the reflection penalty on 8 x 152,064 logits and the
    answer perplexity over 8 x 32 answer tokens."""
    wl = I.WORKLOADS["32b64k"]
    units = [(0, 0, 0), (17, 3, 5), (40, 6, 7), (63, 7, 2)]
    ci, cache = _run_workload(wl, units, decode_steps=3, check_steps={0, 2})
    assert cache.shape == (64, 8, 8, 65536 + wl.decode_steps, 128)
    del cache, ci
    torch.cuda.empty_cache()
    dev = torch.device("cuda")
    V = wl.vocab
    reward = np.array([0.1, 0.4, 0.41, 0.6, 0.79, 0.8, 0.95, 1.0], dtype=np.float32)
    z0 = I.make_logits(8, V, seed=wl.seed + 17)
    ids = I.make_reflection_ids(wl.n_reflection_ids, V, seed=wl.seed + 19)
    z = z0.to(dev)
    B.reco_logit_penalty(z, torch.from_numpy(ids).to(dev), torch.from_numpy(reward).to(dev), 0.4, 0.8, 0.0, 1.0, 3.0)
    ref = oracle.logit_penalty(z0.numpy(), ids, reward, 0.4, 0.8, 0.0, 1.0, 3.0)
    assert z.cpu().numpy().tobytes() == ref.tobytes()
    logits = I.make_logits(8 * 32, V, seed=wl.seed + 23, shape=(8, 32, V))
    tok = I.make_answer_tokens(8, 32, V, seed=wl.seed + 29)
    logits[2, np.arange(32), tok[2]] += 25.0                 # one confident answer
    ppl, stop = B.reco_answer_ppl(logits.to(dev), torch.from_numpy(tok).to(dev), 1.1)
    rp, rs = oracle.answer_ppl(logits.numpy(), tok, 1.1)
    assert np.abs(np.log(ppl.cpu().numpy().astype(np.float64)) - np.log(rp)).max() <= 1e-5
    assert stop.cpu().numpy().tolist() == rs.astype(int).tolist()
