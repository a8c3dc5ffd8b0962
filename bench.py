#!/usr/bin/env python3
"""Throughput of the reward-coordinated compression hot path on one MI355X.

One step = one pass of the whole path over one batch of synthetic input:
  window scoring (Eq. 2) -> reward-budgeted selection + in-place compaction
  -> `decode_steps` decode-attention calls over all layers (each appending the
  new token), the banded reflection-logit penalty (Eq. 3-4) on every
  generated token's logit row with the next token drawn from softmax(z~)
  (one fused pass over the rows) -> one answer-perplexity probe (Eq. 5-6).
Every step starts from its own pristine copy of the cache, staged in HBM
before the timed region.  Prints one JSON line (rank 0, N = 1).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 7b16k] [--no-cpu-baseline] [--no-extras]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2608_04771_amd import binding as B  # noqa: E402
from paper_2608_04771_amd import inputs as I  # noqa: E402

PEAK_HBM_GBPS = 8000.0          # MI355X HBM3E vendor peak
METRIC = "compress+decode-attn KV tokens/s and achieved HBM GB/s (% of peak), 1 GPU"
TAU_LO, TAU_HI, TAU_P = 0.4, 0.8, 1.1          # Section 4.1
BETAS = (0.0, 1.0, 3.0)                        # penalty per reward band
TEMPERATURE = 1.0                              # sample from softmax(z~) itself
SAMPLE_SEED = 0x5EED
N_REFL = 64
ANSWER_LEN = 32

# HBM traffic of one decode_split_kernel launch on this workload, from two
# rocprofv3 counter passes (FETCH_SIZE, WRITE_SIZE), each scaled by what the
# counter reads for a plain device copy of known size (factors 0.5001 and
# 1.0000).  Valid only for the kernel sources it was taken with: if those
# files change, the figure is reported as null until it is measured again.
DECODE_TRAFFIC = {
    "sources": ("paper_2608_04771_amd/csrc/decode_attn.hip", "paper_2608_04771_amd/csrc/reco_device.hpp",
                "paper_2608_04771_amd/csrc/decode_attn.hpp"),
    "sha256": "c32943c7a959a935db735c184a74d62495d0a4c6a6f2b30369b0685d872f471f",
    "workload": "7b-28L-28q4kv-d128-bf16-L16384",
    "fetch_bytes": 555477303,
    "write_bytes": 817152,
}


def decode_traffic(workload_name: str):
    import hashlib
    h = hashlib.sha256()
    for f in DECODE_TRAFFIC["sources"]:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    if h.hexdigest() != DECODE_TRAFFIC["sha256"] or workload_name != DECODE_TRAFFIC["workload"]:
        return None
    return DECODE_TRAFFIC["fetch_bytes"] + DECODE_TRAFFIC["write_bytes"]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class Workload:
    """Device-resident inputs of one workload plus per-step cache copies."""

    def __init__(self, wl: I.Workload, copies: int, dev):
        self.wl = wl
        ci = I.make_cache(wl)
        self.ci = ci
        self.dev = dev
        log(f"generated cache {tuple(ci.k.shape)} {wl.dtype}")
        k0, v0, l0 = ci.k.to(dev), ci.v.to(dev), ci.length.to(dev)
        self.copies = [(k0.clone(), v0.clone(), l0.clone()) for _ in range(copies)]
        del k0, v0, l0
        self.q_win = ci.q_win.to(dev)
        self.retention = torch.tensor([B.reco_retention_from_reward(float(v)) for v in ci.reward],
                                      dtype=torch.float64, device=dev)
        qs, ks, vs = I.make_decode_inputs(wl, ci, wl.decode_steps)
        self.q = torch.stack(qs).to(dev)
        self.k_new = torch.stack(ks).to(dev)
        self.v_new = torch.stack(vs).to(dev)
        Bsz = len(ci.seq_len)
        V = wl.vocab
        self.logits = I.make_logits(wl.decode_steps * Bsz, V, seed=wl.seed + 17).to(dev).view(wl.decode_steps, Bsz, V)
        self.refl = torch.from_numpy(I.make_reflection_ids(N_REFL, V, seed=wl.seed + 19)).to(dev)
        self.step_reward = torch.from_numpy(ci.reward.astype(np.float32)).to(dev)
        # every generated token of the step is penalised with the band of the step's reward
        self.row_reward = self.step_reward.repeat(wl.decode_steps).contiguous()
        self.ans_logits = I.make_logits(Bsz * ANSWER_LEN, V, seed=wl.seed + 23,
                                        shape=(Bsz, ANSWER_LEN, V)).to(dev)
        self.ans_tok = torch.from_numpy(I.make_answer_tokens(Bsz, ANSWER_LEN, V, seed=wl.seed + 29)).to(dev)
        NL, Bsz, H, Cap, D = self.copies[0][0].shape
        self.shape = (NL, Bsz, H, Cap, D)
        c = B.KVCache(*self.copies[0])
        self.scores = torch.zeros((NL, Bsz, H, Cap), dtype=torch.float32, device=dev)
        self.kept = torch.zeros((NL, Bsz, H, Cap), dtype=torch.int32, device=dev)
        self.ws_score = torch.empty(B.score_workspace_size(c, wl.n_q_heads, wl.window), dtype=torch.uint8, device=dev)
        self.ws_sel = torch.empty(B.select_compact_workspace_size(c), dtype=torch.uint8, device=dev)
        self.ws_dec = B.decode_workspace(c, wl.n_q_heads)
        self.ws_ppl = torch.empty(B.answer_ppl_workspace_size(Bsz, ANSWER_LEN, V), dtype=torch.uint8, device=dev)
        self.ws_smp = torch.empty(B.penalty_sample_workspace_size(wl.decode_steps * Bsz, V), dtype=torch.uint8,
                                  device=dev)
        self.tokens = torch.empty(wl.decode_steps * Bsz, dtype=torch.int32, device=dev)
        # (max, sum) softmax statistics of every decode query, kept for one-pass scoring
        self.stats = torch.empty((wl.decode_steps, NL, Bsz, wl.n_q_heads, 2), dtype=torch.float32, device=dev)
        self.out = torch.empty_like(self.q[0])
        self.lse = torch.empty(self.q.shape[1:4], dtype=torch.float32, device=dev)
        self.ppl = torch.empty(Bsz, dtype=torch.float32, device=dev)
        self.stop = torch.empty(Bsz, dtype=torch.int32, device=dev)
        self.dev_err = torch.zeros(1, dtype=torch.int32, device=dev)
        self.side = torch.cuda.Stream(device=dev)       # default priority

    def step(self, i, ev=None):
        """One pass of the hot path on cache copy i.  The penalise-and-sample
        pass over the logit rows of all decode steps (one call, row = token x
        sequence) runs on a side stream, as it is independent of the
        attention, and joins the main stream before the answer probe.  `ev`
        optionally collects HIP events on the main stream around the phases."""
        wl = self.wl
        cache = B.KVCache(*self.copies[i])
        main = torch.cuda.current_stream()
        if ev is not None:
            ev["c0"].record()
        B.reco_score(cache, self.q_win, wl.window, scores=self.scores, ws=self.ws_score, dev_err=self.dev_err)
        if ev is not None:
            ev["c1"].record()
        B.reco_select_compact(cache, self.scores, self.retention, wl.window, kept_idx=self.kept, ws=self.ws_sel,
                              dev_err=self.dev_err)
        if ev is not None:
            ev["c2"].record()
        self.side.wait_stream(main)
        with torch.cuda.stream(self.side):
            if ev is not None:
                ev["s0"].record()
            B.reco_penalty_sample(self.logits.view(-1, self.logits.shape[-1]), self.refl, self.row_reward, TAU_LO,
                                  TAU_HI, *BETAS, TEMPERATURE, SAMPLE_SEED, i, tokens=self.tokens, ws=self.ws_smp,
                                  dev_err=self.dev_err)
            if ev is not None:
                ev["s1"].record()
        for s in range(wl.decode_steps):
            B.reco_decode_attn(cache, self.q[s], self.k_new[s], self.v_new[s], out=self.out, lse=self.lse,
                               ws=self.ws_dec, dev_err=self.dev_err, row_stats=self.stats[s])
        if ev is not None:
            ev["d1"].record()
        main.wait_stream(self.side)
        if ev is not None:
            ev["p0"].record()
        B.reco_answer_ppl(self.ans_logits, self.ans_tok, TAU_P, ppl=self.ppl, stop=self.stop, ws=self.ws_ppl,
                          dev_err=self.dev_err)
        if ev is not None:
            ev["p1"].record()


def score_after_decode(w: Workload, i: int, reps: int = 5):
    """Scoring of the post-decode cache of copy i with its last `window`
    decode tokens as the window, once with the two-pass kernels and once fed
    with the statistics those decode calls wrote (no compression happened
    since, so both compute Eq. 2 over the same keys).  Outside the timed step."""
    wl = w.wl
    win = wl.window
    cache = B.KVCache(*w.copies[i])
    q_win = w.q[-win:].permute(1, 2, 3, 0, 4).contiguous()          # [NL][B][Hq][w][D]
    st_win = w.stats[-win:].permute(1, 2, 3, 0, 4).contiguous()      # [NL][B][Hq][w][2]
    a, b = torch.zeros_like(w.scores), torch.zeros_like(w.scores)
    E = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    out = {}
    for name, stats, dst in (("two_pass", None, a), ("stats_fed", st_win, b)):
        B.reco_score(cache, q_win, win, scores=dst, ws=w.ws_score, dev_err=w.dev_err, row_stats=stats)
        e0, e1 = E(), E()
        e0.record()
        for _ in range(reps):
            B.reco_score(cache, q_win, win, scores=dst, ws=w.ws_score, dev_err=w.dev_err, row_stats=stats)
        e1.record()
        torch.cuda.synchronize()
        out[name + "_ms"] = e0.elapsed_time(e1) / reps
    rel = ((b - a).abs() / a.clamp_min(1e-30)).masked_fill(a <= 1e-20, 0.0)
    out["max_rel_diff"] = float(rel.max().item())
    out["cache_rows"] = int(cache.length.max().item())
    return out


def decode_per_layer_graph(w: Workload, i: int, reps: int = 20):
    """The model-faithful form of one decode step: one reco_decode_attn call
    per layer (as a model interleaves them with its other layers), the
    NL calls captured once in a HIP graph and replayed.  Runs on the
    post-decode cache of copy i (each replay appends one more token),
    outside the timed step."""
    wl = w.wl
    NL = w.shape[0]
    cache = B.KVCache(*w.copies[i])
    q, kn, vn = w.q[0], w.k_new[0], w.v_new[0]
    ws = torch.empty(B.decode_attn_workspace_size(cache, wl.n_q_heads, 1), dtype=torch.uint8, device=q.device)
    out = torch.empty_like(q)
    lse = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device)

    def one_step():
        for l in range(NL):
            B.reco_decode_attn(cache, q[l:l + 1], kn[l:l + 1], vn[l:l + 1], out=out[l:l + 1], lse=lse[l:l + 1],
                               layer0=l, n_layers=1, ws=ws, dev_err=w.dev_err)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        one_step()                                     # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        one_step()
    g.replay()
    torch.cuda.synchronize()
    E = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    e0, e1 = E(), E()
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return {"us_per_decode_step": e0.elapsed_time(e1) * 1e3 / reps, "calls_per_step": NL,
            "cache_rows": int(cache.length.max().item())}


def copy_bandwidth(w: Workload):
    """Context: a plain device-to-device copy of one cache's K (read + write)."""
    src = w.copies[0][0]
    dst = torch.empty_like(src)
    dst.copy_(src)
    E = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    e0, e1 = E(), E()
    e0.record()
    for _ in range(5):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    return 2 * src.numel() * src.element_size() * 5 / (e0.elapsed_time(e1) * 1e-3) / 1e9


def make_events():
    E = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    return {"c0": E(), "c1": E(), "c2": E(), "d1": E(), "p0": E(), "p1": E(), "s0": E(), "s1": E()}


def algorithmic_bytes(w: Workload, m: np.ndarray, moved_rows: int):
    """Bytes the method has to move (not what an implementation re-reads)."""
    wl = w.wl
    NL, Bsz, H, Cap, D = w.shape
    e = wl.elem_bytes
    Hq = wl.n_q_heads
    L = w.ci.seq_len                                  # [B]
    units_L = NL * H * int(L.sum())
    score = units_L * D * e + NL * Bsz * Hq * wl.window * D * e + units_L * 4
    select = units_L * 4 + int(m.sum()) * 4
    compact = moved_rows * 2 * 2 * D * e
    dec = []
    for s in range(wl.decode_steps):
        rows = int((m + s + 1).sum())                 # keys attended (cached + new) over all units
        dec.append(rows * 2 * D * e + 2 * NL * Bsz * Hq * D * e + NL * Bsz * Hq * 4 + 2 * m.size * D * e)
    penalty = wl.decode_steps * Bsz * (wl.vocab * 4 + N_REFL * 4 + 4)   # read the row, write R and the token
    ppl = Bsz * ANSWER_LEN * wl.vocab * 4
    return {"score": score, "select": select, "compact": compact, "decode": dec, "penalty": penalty, "ppl": ppl}


def kv_tokens(w: Workload, m_seq: np.ndarray):
    """KV tokens per step: one cached position of one sequence in one layer."""
    wl = w.wl
    NL = w.shape[0]
    compress = NL * int(w.ci.seq_len.sum())
    decode = sum(NL * int((m_seq + s + 1).sum()) for s in range(wl.decode_steps))
    return compress, decode


def cpu_baseline(w: Workload, comp_budget_s: float = 8.0, dec_budget_s: float = 10.0):
    """The CPU oracle as it stands, timed on a bounded sample of the workload:
    the compression of whole layers (all their units) and decode steps of one
    layer spread over the decode range, until each phase has used its time
    budget; the per-phase rates are then scaled to one full step."""
    import oracle
    from threadpoolctl import threadpool_info, threadpool_limits
    # Host cores this process may run on; the oracle's BLAS pool is set to
    # that count, capped by the job's thread budget (OMP_NUM_THREADS) where
    # one is set, so that it never oversubscribes the cores it was given.
    affinity = len(os.sched_getaffinity(0))
    budget = int(os.environ.get("OMP_NUM_THREADS", "0") or 0)
    threads = min(affinity, budget) if budget > 0 else affinity
    with threadpool_limits(limits=threads):
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
        res = _cpu_baseline_sample(w, oracle, comp_budget_s, dec_budget_s)
    res["cores"] = int(cores)
    res["affinity_cores"] = affinity
    return res


def _cpu_baseline_sample(w: Workload, oracle, comp_budget_s: float, dec_budget_s: float):
    wl = w.wl
    ci = w.ci
    NL, Bsz, H, Cap, D = w.shape
    scale = 1.0 / math.sqrt(D)
    r = [oracle.retention_from_reward(float(v)) for v in ci.reward]
    cpu_s = 0.0                      # process CPU time (all threads) inside the timed oracle calls
    t_comp, n_comp = 0.0, 0
    comp = None
    while n_comp < NL and (n_comp == 0 or t_comp < comp_budget_s):
        Kl, Vl = I.to_f64(ci.k[n_comp])[None], I.to_f64(ci.v[n_comp])[None]
        Ql = I.to_f64(ci.q_win[n_comp])[None]
        lens = ci.length.numpy()[n_comp:n_comp + 1].astype(np.int64)
        c0, t0 = time.process_time(), time.perf_counter()
        res = oracle.compress_cache(Kl, Vl, lens, Ql, r, wl.window, scale)
        t_comp += time.perf_counter() - t0
        cpu_s += time.process_time() - c0
        comp = comp or res
        n_comp += 1
    _, _, K2, V2, l2 = comp
    qs, _, _ = I.make_decode_inputs(wl, ci, 1)
    q1 = I.to_f64(qs[0][:1])
    order = list(range(0, wl.decode_steps, max(1, wl.decode_steps // 32)))
    t_dec, n_dec = 0.0, 0
    while n_dec < 4096 and (n_dec == 0 or t_dec < dec_budget_s):
        s_idx = order[n_dec % len(order)]
        # Decode step s_idx attends over m + s_idx + 1 rows (the cached ones and
        # the appended token); the sample attends over the same number of rows
        # without writing the appended row, so the cache needs no copy.
        lens_s = l2 + s_idx + 1
        c0, t0 = time.process_time(), time.perf_counter()
        oracle.decode_cache(K2, V2, lens_s, q1, scale)
        t_dec += time.perf_counter() - t0
        cpu_s += time.process_time() - c0
        n_dec += 1
    # Average number of busy host threads over the timed oracle calls.
    busy = cpu_s / max(t_comp + t_dec, 1e-9)
    m_seq = l2[0, :, 0]
    comp_tok, dec_tok = kv_tokens(w, m_seq)
    est_step_s = NL * t_comp / n_comp + NL * wl.decode_steps * t_dec / n_dec
    return {"value": (comp_tok + dec_tok) / est_step_s, "unit": "KV tokens/s",
            "avg_busy_threads": round(busy, 2), "kind": "oracle",
            "sample": (f"{n_comp} of {NL} layers compressed ({n_comp * H * Bsz} units, {t_comp:.2f} s) and "
                       f"{n_dec} decode steps of 1 layer spread over the {wl.decode_steps}-step range "
                       f"({t_dec:.2f} s); per-phase rates scaled to one full step "
                       f"({est_step_s:.1f} s estimated)")}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    # The batch, 32B and trajectory workloads do not fit this bench's one
    # pristine cache copy per step; the full-size GPU tests measure them.
    ap.add_argument("--workload", default="7b16k", choices=["7b16k", "tiny"])
    ap.add_argument("--no-cpu-baseline", dest="cpu_baseline", action="store_false")
    ap.add_argument("--no-extras", dest="extras", action="store_false",
                    help="skip the measurements made after the timed steps (for profiler runs)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the hot path is built and timed on a single MI355X "
              "(units of (layer, sequence, KV head) would shard across GPUs with no exchange, but no "
              "multi-GPU path is built); run it with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    B.load_library()
    wl = I.WORKLOADS[args.workload]
    copies = args.warmup + args.steps
    w = Workload(wl, copies, dev)
    torch.cuda.synchronize()
    log(f"staged {copies} cache copies; warmup {args.warmup}")
    for i in range(args.warmup):
        w.step(i)
    torch.cuda.synchronize()
    if w.dev_err.item() != 0:
        raise RuntimeError(f"device error {w.dev_err.item()}")
    log("warmup done; timing")
    evs = [make_events() for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        w.step(args.warmup + i, evs[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step")
    score_fed = per_layer = copy_gbps = None
    if args.extras:
        score_fed = score_after_decode(w, args.warmup + args.steps - 1)
        per_layer = decode_per_layer_graph(w, args.warmup + args.steps - 1)
        copy_gbps = copy_bandwidth(w)

    # Sizes of this workload's steps (identical for every copy).
    lens_after = w.copies[args.warmup][2].cpu().numpy()
    m = lens_after.astype(np.int64) - wl.decode_steps          # kept rows per unit
    kept = w.kept.cpu().numpy()
    moved = 0
    for u in np.ndindex(*m.shape):
        mu = int(m[u])
        moved += int((kept[u][:mu] != np.arange(mu)).sum())
    ab = algorithmic_bytes(w, m, moved)
    step_bytes = ab["score"] + ab["select"] + ab["compact"] + sum(ab["decode"]) + ab["penalty"] + ab["ppl"]
    comp_tok, dec_tok = kv_tokens(w, m[0, :, 0])
    tok = comp_tok + dec_tok

    # The decode calls of a step run back to back on the main stream between
    # events c2 and d1 (the penalties overlap on the side stream), so their
    # average duration is that interval over the number of calls.
    dec_loop_ms = np.array([ev["c2"].elapsed_time(ev["d1"]) for ev in evs])
    comp_ms = np.array([ev["c0"].elapsed_time(ev["c2"]) for ev in evs])
    score_ms = np.array([ev["c0"].elapsed_time(ev["c1"]) for ev in evs])
    sel_ms = np.array([ev["c1"].elapsed_time(ev["c2"]) for ev in evs])
    ppl_ms = np.array([ev["p0"].elapsed_time(ev["p1"]) for ev in evs])
    smp_ms = np.array([ev["s0"].elapsed_time(ev["s1"]) for ev in evs])
    dec_bytes_mean = float(np.mean(ab["decode"]))
    dec_avg_ms = float(dec_loop_ms.mean()) / wl.decode_steps
    achieved = dec_bytes_mean / (dec_avg_ms * 1e-3) / 1e9

    res = {
        "metric": METRIC,
        "value": tok / (ms_per_step * 1e-3),
        "unit": "KV tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "n_layers": wl.n_layers, "batch": int(len(w.ci.seq_len)),
                   "q_heads": wl.n_q_heads, "kv_heads": wl.n_kv_heads, "head_dim": wl.head_dim,
                   "cache_len": int(w.ci.seq_len.max()), "window": wl.window, "decode_steps": wl.decode_steps,
                   "retention": float(w.retention[0].item()), "kept_rows": int(m.max()), "vocab": wl.vocab,
                   "seed": wl.seed},
        "achieved_GBps": step_bytes / (ms_per_step * 1e-3) / 1e9,
        "pct_of_peak_hbm": 100.0 * step_bytes / (ms_per_step * 1e-3) / 1e9 / PEAK_HBM_GBPS,
        "algorithmic_bytes_per_step": step_bytes,
        "kv_tokens_per_step": {"compress": comp_tok, "decode": dec_tok},
        "compress_algorithmic_bytes": {"score": ab["score"], "select": ab["select"], "compact": ab["compact"],
                                       "compact_moved_rows": moved},
        "phase_ms": {"score": float(score_ms.mean()), "select_compact": float(sel_ms.mean()),
                     "compress": float(comp_ms.mean()), "decode_call": dec_avg_ms,
                     "decode_calls_total": float(dec_loop_ms.mean()), "answer_ppl": float(ppl_ms.mean())},
        "score_after_decode": score_fed,
        "decode_per_layer_graph": per_layer,
        "penalty_sample": {"ms_per_step": float(smp_ms.mean()), "rows_per_step": int(w.tokens.numel()),
                           "us_per_row": float(smp_ms.mean()) * 1e3 / int(w.tokens.numel()),
                           "stream": "side (overlaps the decode calls)"},
        "copy_GBps_context": copy_gbps,
        "roofline": {"kernel": "reco_decode_attn (decode_split_kernel + decode_merge_kernel)", "bound": "hbm",
                     "achieved": achieved, "peak": PEAK_HBM_GBPS, "unit": "GB/s", "frac": achieved / PEAK_HBM_GBPS,
                     "traffic": decode_traffic(wl.name), "traffic_unit": "bytes per decode_split_kernel launch",
                     "algorithmic_bytes_per_launch": dec_bytes_mean},
    }
    if args.cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        res["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
