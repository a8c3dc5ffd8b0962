"""Step-wise compression at the 32B-shaped full size (Section 3.2: the cache is
compressed again whenever it has grown by S tokens since the last
compression, with a retention set by the latest step's reward).

64 layers x 8 sequences x 8 KV heads (GQA 5), 65,536 cached tokens, window
32, four rounds of (compress -> 64 decode steps), every call over all layers:
* round 1 scores with the two-pass kernels and the workload's window queries;
* rounds 2-4 score in one pass over K: the window is the last 32 decode
  queries of the previous round, with the softmax statistics their decode
  calls wrote (no compression happened since they were decoded, so those
  statistics are Eq. 2's normalisers);
* each round has its own per-sequence reward v ~ Beta(2, 2) -> r(v), and
  compresses a cache that was compacted and then appended to.

Every round checks, on sampled units, the scores against the oracle (and the
near-theta precision), the kept sets (ties excused), the gathered rows bit for
bit against a snapshot taken before the compression, and decode outputs and
log-sum-exps at the first and last step; on all 4,096 units it checks the
lengths and the mass conservation of the scores (each unit's scores sum to
G * w) after every compression, the lengths again after the decode steps,
and the last decode call of each round against a plain PyTorch fp32
attention on the device.  The phase times of every round are printed."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import (SCORE_RTOL, assert_decode_all_units, assert_decode_close, assert_lse_close,
                         assert_mass_conserved, assert_theta_precision, f64, kept_sets_match)
from paper_2608_04771_amd import binding as B
from paper_2608_04771_amd import inputs as I

pytestmark = pytest.mark.gpu

ROUNDS = 4
UNITS = [(0, 0, 0), (17, 3, 5), (40, 6, 7), (63, 7, 2)]


def test_32b_64k_four_rounds_stepwise():
    wl = I.WORKLOADS["32b64k"]
    steps, w, G = wl.decode_steps, wl.window, wl.group
    dev = torch.device("cuda")
    print(f"{wl.name}: {ROUNDS} rounds x (compress -> {steps} decode)", flush=True)
    ci = I.make_cache(wl, device=dev, capacity=int(wl.lengths[0]) + ROUNDS * steps)
    cache = B.KVCache(ci.k, ci.v, ci.length)
    NL, Bsz, H, Cap, D = cache.shape
    Hq = wl.n_q_heads
    scale = 1.0 / np.sqrt(D)
    rewards = I.make_rewards("beta22", ROUNDS, Bsz, seed=wl.seed + 31)
    dev_err = torch.zeros(1, dtype=torch.int32, device=dev)
    scores = torch.zeros((NL, Bsz, H, Cap), dtype=torch.float32, device=dev)
    kept = torch.full((NL, Bsz, H, Cap), -1, dtype=torch.int32, device=dev)
    ws_score = torch.empty(B.score_workspace_size(cache, Hq, w), dtype=torch.uint8, device=dev)
    ws_sel = torch.empty(B.select_compact_workspace_size(cache), dtype=torch.uint8, device=dev)
    ws_dec = B.decode_workspace(cache, Hq)
    out = torch.empty((NL, Bsz, Hq, D), dtype=ci.k.dtype, device=dev)
    lse = torch.empty((NL, Bsz, Hq), dtype=torch.float32, device=dev)
    stats = torch.empty((steps, NL, Bsz, Hq, 2), dtype=torch.float32, device=dev)
    q_win, row_stats = ci.q_win, None
    E = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731

    for rnd in range(ROUNDS):
        lens0 = cache.length.cpu().numpy()
        r = np.array([oracle.retention_from_reward(float(v)) for v in rewards[rnd]])
        snap = {u: (int(lens0[u]), f64(cache.k[u][:int(lens0[u])]), f64(cache.v[u][:int(lens0[u])]))
                for u in UNITS}
        qw = {u: f64(q_win[u[0], u[1], u[2] * G:(u[2] + 1) * G]) for u in UNITS}
        print(f"round {rnd + 1}: compress {'one-pass' if row_stats is not None else 'two-pass'} over "
              f"{int(lens0.sum())} rows, r = {np.round(r, 4).tolist()}", flush=True)
        ev = [E() for _ in range(5)]
        ev[0].record()
        B.reco_score(cache, q_win, w, scores=scores, ws=ws_score, dev_err=dev_err, row_stats=row_stats)
        ev[1].record()
        B.reco_select_compact(cache, scores, torch.from_numpy(r).to(dev), w, kept_idx=kept, ws=ws_sel,
                              dev_err=dev_err)
        ev[2].record()
        torch.cuda.synchronize()
        assert dev_err.item() == 0
        assert_mass_conserved(scores, torch.from_numpy(lens0.astype(np.int64)), G, w, f"round {rnd + 1}")
        score_ms, sel_ms = ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2])
        lens1 = cache.length.cpu().numpy()
        for u in np.ndindex(NL, Bsz, H):
            assert lens1[u] == oracle.kept_count(int(lens0[u]), w, float(r[u[1]])), (rnd, u)
        for u in UNITS:
            L, K0, V0 = snap[u]
            s_or = oracle.score_unit(K0, qw[u], scale)
            s_gpu = scores[u][:L].cpu().numpy().astype(np.float64)
            assert (np.abs(s_gpu - s_or) / s_or).max() <= SCORE_RTOL, (rnd, u)
            assert_theta_precision(s_gpu, s_or, L, w, float(r[u[1]]), f"round {rnd + 1} unit {u}")
            kk = kept[u].cpu().numpy()
            ok, msg = kept_sets_match(kk, s_or, L, w, float(r[u[1]]))
            assert ok, (rnd, u, msg)
            m = int(lens1[u])
            np.testing.assert_array_equal(f64(cache.k[u][:m]), K0[kk[:m]])
            np.testing.assert_array_equal(f64(cache.v[u][:m]), V0[kk[:m]])
        del snap

        qs, ks, vs = I.make_decode_inputs(wl, ci, steps, seed_offset=rnd + 1, device=dev)
        for s in range(steps):
            if s == 1:
                ev[3].record()                       # steps 1 .. steps-1 run back to back: timed
            B.reco_decode_attn(cache, qs[s], ks[s], vs[s], out=out, lse=lse, ws=ws_dec, dev_err=dev_err,
                               row_stats=stats[s])
            if s in (0, steps - 1):
                if s == steps - 1:
                    ev[4].record()
                torch.cuda.synchronize()
                if s == steps - 1:
                    assert_decode_all_units(cache, qs[s], out, lse, torch.from_numpy(lens1.astype(np.int64)) + s + 1,
                                            scale, f"round {rnd + 1} step {s}")
                for u in UNITS:
                    l, b, h = u
                    n = int(lens1[u]) + s + 1                        # the call appended row n - 1
                    ref, rl = oracle.decode_unit(f64(cache.k[u][:n]), f64(cache.v[u][:n]), n,
                                                 f64(qs[s][l, b, h * G:(h + 1) * G]), scale)
                    assert_decode_close(out[l, b, h * G:(h + 1) * G], ref, "bf16", f"round {rnd + 1} step {s} {u}")
                    assert_lse_close(lse[l, b, h * G:(h + 1) * G], rl, "bf16", f"round {rnd + 1} step {s} {u}")
        torch.cuda.synchronize()
        assert dev_err.item() == 0
        assert (cache.length.cpu().numpy() == lens1 + steps).all()
        dec_ms = ev[3].elapsed_time(ev[4]) / (steps - 1)
        # K and V rows read by an average timed call (cached rows plus the new one)
        rows = int(lens1.sum()) + NL * Bsz * H * (steps // 2 + 1)
        k_pass = int(lens0.sum()) * D * 2
        print(f"round {rnd + 1}: score {score_ms:.2f} ms ({k_pass / score_ms / 1e9:.2f} TB/s of one K pass), "
              f"select+compact {sel_ms:.2f} ms, decode call {dec_ms:.2f} ms "
              f"({rows * 2 * D * 2 / dec_ms / 1e9:.2f} TB/s), kept {int(lens1.max())} rows per unit", flush=True)
        # The next round's window: the last w decode queries, [NL][B][Hq][w][D],
        # with the statistics their decode calls wrote.
        q_win = torch.stack(qs[-w:], dim=3).contiguous()
        row_stats = stats[-w:].permute(1, 2, 3, 0, 4).contiguous()
        del qs, ks, vs
