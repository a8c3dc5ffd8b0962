"""Host control plane of reward-coordinated decoding (Section 3), on the HIP kernels.

The paper's loop, per completed reasoning step i with process reward v_i:

* reward-driven retention (Section 3.2, Eq. 1 and its schedule): compress
  when L - L_{i-1} >= S, down to m_i = lambda_i * L rows, where lambda_i
  follows v_i measured against the trajectory's reward history (or the fixed
  map r = clamp(1 - v/2, 0.3, 1));
* attention-guided selection (Eq. 2) over the w most recent queries;
* the reward band of the just-completed step sets the reflection-token
  penalty applied to every logit row of the next step (Eq. 3-4), and the
  next token is drawn from the softmax of the penalised row;
* two consecutive top-band rewards trigger the answer probe, whose
  perplexity decides the stop (Eq. 5-6).

Scoring reuses the softmax statistics that decode attention wrote for the
window tokens (one pass over K instead of two) whenever every window token
was decoded after the last compression, so that the keys each of them saw
are exactly the keys it sees now.

Policy variants on the same kernels: delta = 0 (one uniform retention, the
paper's own ablation of Eq. 1), per-layer budgets (`layer_spread`, a
retention falling linearly with depth that averages r) and pooled scores
(`pool_kernel`, max or mean pooling of the prefix scores before the top-k),
the last two after the eviction methods the paper cites in Section 1.

`RewardSchedule` holds the pure host bookkeeping (reward history, retention,
compression trigger, probe trigger) and runs without a GPU.  `RecoDecoder`
drives the kernels through the binding: it keeps the window queries in a ring
buffer on the device, calls reco_decode_attn and reco_logit_penalty (or the
fused reco_penalty_sample) per token and reco_score / reco_select_compact at
step boundaries.  The two per-token calls go through the binding's prepared
forms, which check the decoder's fixed buffers once and each token's tensors
on every call.  All arithmetic of the method runs in the library; this
module decides when, and moves data.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import torch

from . import binding as B


@dataclasses.dataclass
class RecoPolicy:
    """Hyper-parameters of the loop.  Defaults are the fixed set of Section 4.1
    (lambda = 0.25, delta = 0.1, w = 32, tau_l = 0.4, tau_h = 0.8, tau_p = 1.1);
    `retention="clamp"` selects r = clamp(1 - v/2, lo, hi) instead of Eq. 1."""
    retention: str = "eq1"           # "eq1" | "clamp"
    lam: float = 0.25
    delta: float = 0.1
    lo: float = 0.3
    hi: float = 1.0
    window: int = 32
    interval: int = 0                # S: compress once the cache grew by S tokens (0: every step boundary)
    tau_lo: float = 0.4
    tau_hi: float = 0.8
    tau_p: float = 1.1
    betas: Sequence[float] = (0.0, 1.0, 3.0)   # penalty in the low / middle / high band
    layer_spread: float = 0.0        # per-layer budgets: r_l from r(1 + spread) at layer 0 to r(1 - spread)
    pool_kernel: int = 1             # score pooling before selection (1: none; odd, <= 65)
    pool_mode: str = "max"           # "max" | "mean"
    stats_fed: bool = True           # score with the window tokens' decode statistics when they are exact


class RewardSchedule:
    """Per-sequence host state: reward history, cache length bookkeeping (one
    length per layer) and the two triggers.  Lengths follow the same fp64
    kept-count rule as the select kernel, so no device read-back is needed."""

    def __init__(self, policy: RecoPolicy, prompt_len: int, n_layers: int = 1):
        self.policy = policy
        self.n_layers = int(n_layers)
        self.rewards: List[float] = []
        self.lengths = [int(prompt_len)] * self.n_layers   # L per layer
        self.length_at_compress = int(prompt_len)          # layer 0's L after the last compression
        self.grown = 0                                     # tokens appended since the last compression
        self.top_streak = 0

    @property
    def length(self) -> int:
        """Layer 0's cache length (every layer's when the budget is uniform)."""
        return self.lengths[0]

    def retention(self) -> float:
        p = self.policy
        v = self.rewards[-1]
        if p.retention == "clamp":
            return B.reco_retention_from_reward(v, p.lo, p.hi)
        return B.reco_retention_eq1(self.rewards, p.lam, p.delta)

    def layer_retentions(self, r: float) -> List[float]:
        """The retention of every layer for sequence-level retention r."""
        if self.policy.layer_spread == 0.0:
            return [r] * self.n_layers
        return [B.reco_layer_retention(r, l, self.n_layers, self.policy.layer_spread) for l in range(self.n_layers)]

    def token_appended(self, n: int = 1):
        self.lengths = [L + n for L in self.lengths]
        self.grown += n

    def end_step(self, reward: float):
        """Record v_i.  Returns (compress, r, probe): whether the cache is due
        for compression (grown by >= S since the last one), the retention to
        use, and whether the answer probe is due (v >= tau_h twice in a row)."""
        self.rewards.append(float(reward))
        p = self.policy
        self.top_streak = self.top_streak + 1 if reward >= p.tau_hi else 0
        probe = self.top_streak >= 2
        compress = self.grown >= max(1, p.interval)
        r = self.retention()
        return compress, r, probe

    def compressed(self, r: float):
        w = self.policy.window
        self.lengths = [B.reco_kept_count(L, w, rl) for L, rl in zip(self.lengths, self.layer_retentions(r))]
        self.length_at_compress = self.lengths[0]
        self.grown = 0


class RecoDecoder:
    """Drives one batch of sequences through decode steps and step-boundary
    compressions.  All sequences share step boundaries (one schedule per
    sequence; their rewards may differ).

    cache      : KVCache holding the prompt's K/V (length = prompt length)
    n_q_heads  : query heads (GQA group = n_q_heads / n_kv_heads)
    prompt_q   : [NL][B][Hq][w][D] queries of the last w prompt tokens
    refl_ids   : int32 device tensor of reflection-token ids (the set R)
    """

    def __init__(self, cache: B.KVCache, n_q_heads: int, policy: RecoPolicy, prompt_q: torch.Tensor,
                 refl_ids: Optional[torch.Tensor] = None, record_kept: bool = False):
        NL, Bsz, H, Cap, D = cache.shape
        w = policy.window
        if tuple(prompt_q.shape) != (NL, Bsz, n_q_heads, w, D):
            raise ValueError("prompt_q must be [NL][B][Hq][w][D]")
        self.cache, self.policy, self.hq = cache, policy, n_q_heads
        dev = cache.k.device
        prompt_len = int(cache.length[0, 0, 0].item())
        self.sched = [RewardSchedule(policy, prompt_len, NL) for _ in range(Bsz)]
        # slot t % w holds the query of token t, [w][NL][B][Hq][D] (each slot
        # contiguous, so a caller can write the next query straight into it)
        self.ring = prompt_q.permute(3, 0, 1, 2, 4).contiguous()
        # slot t % w holds the (max, sum) decode statistics of token t, [w][NL][B][Hq][2]
        self.stats_ring = torch.zeros((w, NL, Bsz, n_q_heads, 2), dtype=torch.float32, device=dev)
        self.last_score_stats_fed = False
        self.count = prompt_len                           # tokens seen (absolute position of the next one)
        self.refl = refl_ids
        self.band_reward = torch.zeros(Bsz, dtype=torch.float32, device=dev)   # no penalty before the first reward
        self.ws_dec = B.decode_workspace(cache, n_q_heads)
        self.ws_score = torch.empty(B.score_workspace_size(cache, n_q_heads, w), dtype=torch.uint8, device=dev)
        self.ws_sel = torch.empty(B.select_compact_workspace_size(cache), dtype=torch.uint8, device=dev)
        self.scores = torch.zeros((NL, Bsz, H, Cap), dtype=torch.float32, device=dev)
        self.kept = torch.zeros((NL, Bsz, H, Cap), dtype=torch.int32, device=dev) if record_kept else None
        per_layer = policy.layer_spread != 0.0
        self.retention = torch.ones((NL, Bsz) if per_layer else (Bsz,), dtype=torch.float64, device=dev)
        self.pooled = torch.zeros_like(self.scores) if policy.pool_kernel > 1 else None
        self.dev_err = torch.zeros(1, dtype=torch.int32, device=dev)
        self.out = torch.empty((NL, Bsz, n_q_heads, D), dtype=cache.k.dtype, device=dev)
        self.lse = torch.empty((NL, Bsz, n_q_heads), dtype=torch.float32, device=dev)
        self.tokens = torch.empty(Bsz, dtype=torch.int32, device=dev)
        self.ws_smp = None
        self.smp_shape = None                             # (rows, vocab) the sampling workspace was sized for
        # Positions 0..prompt_len-1 are in the cache; the ring's slots hold
        # prompt positions prompt_len - w .. prompt_len - 1 in order, i.e. the
        # slot of position p is p % w once rotated into place.
        shift = prompt_len % w
        if shift:
            self.ring = torch.roll(self.ring, shifts=shift, dims=0).contiguous()
        # The per-token calls, with their fixed buffers checked once here.
        self._decode_call = B.PreparedDecode(cache, n_q_heads, self.out, self.lse, self.ws_dec, self.dev_err)
        self._sample_call = None

    def query_slot(self) -> torch.Tensor:
        """The ring slot of the next token's query, [NL][B][Hq][D]: a caller
        that writes the query here saves decode() the copy."""
        return self.ring[self.count % self.policy.window]

    def decode(self, q: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor,
               logits: Optional[torch.Tensor] = None):
        """One generated token: store its query in the window ring (no copy
        when q is query_slot()), attend (appending its K/V) and apply the
        current reflection penalty to its logit rows ([B][vocab], in place).
        Returns (out, lse)."""
        w = self.policy.window
        slot = self.ring[self.count % w]
        if q.data_ptr() != slot.data_ptr():
            if tuple(q.shape) != tuple(slot.shape) or q.dtype != slot.dtype or q.device != slot.device:
                raise ValueError(f"q must be {list(slot.shape)} {slot.dtype} on {slot.device}")
            slot.copy_(q)
        self._decode_call(slot, k_new, v_new, self.stats_ring[self.count % w])
        if logits is not None and self.refl is not None:
            p = self.policy
            B.reco_logit_penalty(logits, self.refl, self.band_reward, p.tau_lo, p.tau_hi, *p.betas,
                                 dev_err=self.dev_err)
        self.count += 1
        for s in self.sched:
            s.token_appended()
        return self.out, self.lse

    def sample(self, logits: torch.Tensor, temperature: float = 1.0, seed: int = 0) -> torch.Tensor:
        """The current reflection penalty on this token's logit rows ([B][vocab],
        in place) and the next token of every sequence drawn from
        softmax(z~ / T) (T = 0: greedy), in one fused pass.  The draw is keyed
        by (seed, tokens seen so far), so call it once per decoded token.
        Returns the tokens [B] int32 (a buffer reused by the next call)."""
        if self.refl is None:
            raise ValueError("sampling with the reflection penalty needs refl_ids")
        if logits.dim() != 2:
            raise ValueError("logits must be [B][vocab]")
        rows, vocab = logits.shape
        if self.smp_shape != (rows, vocab):
            need = B.penalty_sample_workspace_size(rows, vocab)
            if self.ws_smp is None or self.ws_smp.numel() < need:
                self.ws_smp = torch.empty(need, dtype=torch.uint8, device=logits.device)
            self._sample_call = B.PreparedPenaltySample(rows, vocab, self.refl, self.band_reward, self.tokens,
                                                        self.ws_smp, self.dev_err)
            self.smp_shape = (rows, vocab)
        p = self.policy
        return self._sample_call(logits, p.tau_lo, p.tau_hi, *p.betas, temperature, seed, self.count)

    def window_queries(self) -> torch.Tensor:
        """The last w queries in order (row t = position L - w + t)."""
        w = self.policy.window
        return torch.roll(self.ring, shifts=-(self.count % w), dims=0).permute(1, 2, 3, 0, 4).contiguous()

    def window_stats(self) -> torch.Tensor:
        """Decode statistics of the last w tokens in order, [NL][B][Hq][w][2]."""
        w = self.policy.window
        return torch.roll(self.stats_ring, shifts=-(self.count % w), dims=0).permute(1, 2, 3, 0, 4).contiguous()

    def end_step(self, rewards: Sequence[float]):
        """A reasoning step ended with process rewards v (one per sequence).
        Compresses when due and updates the penalty band for the next step.
        Returns (compressed, probe flags per sequence)."""
        decisions = [s.end_step(v) for s, v in zip(self.sched, rewards)]
        self.band_reward.copy_(torch.tensor([float(v) for v in rewards], dtype=torch.float32))
        probe = [d[2] for d in decisions]
        due = [d[0] for d in decisions]
        if not any(due):
            return False, probe
        # Sequences not due keep everything (r = 1 in every layer keeps every row in place).
        r = [d[1] if d[0] else 1.0 for d in decisions]
        if self.retention.dim() == 2:
            cols = [s.layer_retentions(rr) if d else [1.0] * s.n_layers for s, d, rr in zip(self.sched, due, r)]
            self.retention.copy_(torch.tensor(cols, dtype=torch.float64).T)
        else:
            self.retention.copy_(torch.tensor(r, dtype=torch.float64))
        p = self.policy
        # Decode statistics are exact normalisers only if no compression happened
        # since the oldest window token was decoded.
        fed = p.stats_fed and all(sc.grown >= p.window for sc in self.sched)
        self.last_score_stats_fed = fed
        B.reco_score(self.cache, self.window_queries(), p.window, scores=self.scores, ws=self.ws_score,
                     dev_err=self.dev_err, row_stats=self.window_stats() if fed else None)
        ranked = self.scores
        if self.pooled is not None:
            ranked = B.reco_pool_scores(self.cache, self.scores, p.window, p.pool_kernel, p.pool_mode,
                                        pooled=self.pooled, dev_err=self.dev_err)
        B.reco_select_compact(self.cache, ranked, self.retention, p.window, kept_idx=self.kept,
                              ws=self.ws_sel, dev_err=self.dev_err)
        for s, d, rr in zip(self.sched, due, r):
            if d:
                s.compressed(rr)
        return True, probe

    def answer_ppl(self, logits: torch.Tensor, tokens: torch.Tensor):
        """Eq. 5-6 on a probe answer: (ppl [B], stop [B])."""
        return B.reco_answer_ppl(logits, tokens, self.policy.tau_p, dev_err=self.dev_err)

    def lengths(self) -> List[int]:
        """Layer 0's cache length of every sequence."""
        return [s.length for s in self.sched]

    def layer_lengths(self) -> List[List[int]]:
        """[B][NL] cache lengths."""
        return [list(s.lengths) for s in self.sched]
