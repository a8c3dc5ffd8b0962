"""Seeded synthetic inputs for the reward-coordinated compression hot path.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic (no retention mapping, no scoring, no selection).  Both
the CPU oracle (through the tests and the bench's CPU baseline) and the HIP
path consume exactly the tensors produced here.

Workloads mirror reasoning-shaped KV caches.  The paper evaluates on public
reasoning suites (GSM8K, MATH-500, AMC2023, AIME24/25, GPQA; Section 4.1)
whose chain-of-thought lengths span roughly 1K-15K tokens (Tables 1-2); the
synthetic caches below stand in for them and only reproduce their shapes:

* keys and values ~ N(0, 1); 2% of cached positions per (layer, sequence)
  additionally carry a shared unit direction times 4 (one direction per
  (layer, kv head), added to both K and V) so that they become heavy
  hitters of the attention;
* observation-window queries and decode queries ~ N(0, 1);
* decode tokens are heavy hitters with probability 2%;
* rewards are U(0, 1), Beta(2, 2) or Beta(2, 5) depending on the workload.

Caches are laid out head-major, ``[n_layers][batch][n_kv_heads][capacity][head_dim]``,
so each (layer, sequence, kv head) block is contiguous in memory.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Sequence

import numpy as np
import torch

__all__ = ["Workload", "WORKLOADS", "CacheInputs", "make_cache", "make_decode_inputs",
           "make_logits", "make_reflection_ids", "make_answer_tokens", "make_step_lengths", "make_rewards"]


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape of one synthetic workload.  ``lengths`` gives the cache length of
    every sequence before compression (or a (lo, hi) range when ``ragged``)."""
    name: str
    n_layers: int
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: str                       # "f32" or "bf16"
    lengths: Sequence[int]
    window: int
    decode_steps: int
    reward: str                      # "uniform" | "beta22" | "beta25"
    seed: int
    ragged: bool = False
    hitter_frac: float = 0.02
    hitter_gain: float = 4.0
    vocab: int = 0                   # logit row width for the penalty / answer PPL
    n_reflection_ids: int = 64
    answer_len: int = 32

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def capacity(self) -> int:
        longest = max(self.lengths)
        return longest + self.decode_steps


WORKLOADS = {
    # Tiny parity case: 1 layer, GQA 4, head_dim 64, fp32, 2048 cached tokens,
    # window 32, one compression at v ~ U(0,1), then 64 decode steps.
    "tiny": Workload("tiny-1L-8q2kv-d64-f32-L2048", 1, 1, 8, 2, 64, "f32", (2048,), 32, 64,
                     "uniform", 1000, vocab=4096),
    # 7B-shaped single sequence: 28 layers, 28 query / 4 KV heads, head_dim 128,
    # bf16, 16,384 cached tokens, window 64, one compression at v ~ Beta(2,2),
    # then 256 decode steps over all layers.
    "7b16k": Workload("7b-28L-28q4kv-d128-bf16-L16384", 28, 1, 28, 4, 128, "bf16", (16384,), 64, 256,
                      "beta22", 1001, vocab=152064),
    # 7B-shaped batch: 32 sequences, cache lengths ~ U[4096, 32768], per-sequence
    # rewards ~ Beta(2,2).
    "7b-batch32": Workload("7b-28L-28q4kv-d128-bf16-B32-L4k-32k", 28, 32, 28, 4, 128, "bf16",
                           (4096, 32768), 64, 256, "beta22", 1002, ragged=True, vocab=152064),
    # 8B-shaped full trajectory: 32 layers, 32 query / 8 KV heads, a 512-token
    # prompt, then up to 32,768 generated tokens in steps of Geometric(mean 200)
    # length, rewards ~ Beta(2,5) at every step boundary, 128,256-token vocabulary.
    "8b-trajectory": Workload("8b-32L-32q8kv-d128-bf16-prompt512-gen32768", 32, 1, 32, 8, 128, "bf16", (512,), 32,
                              32768, "beta25", 1003, vocab=128256),
    # 32B-shaped: 64 layers, 40 query / 8 KV heads, batch 8, 65,536 cached tokens.
    "32b64k": Workload("32b-64L-40q8kv-d128-bf16-B8-L65536", 64, 8, 40, 8, 128, "bf16", (65536,), 32, 64,
                       "beta22", 1004, vocab=152064),
}


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


@dataclasses.dataclass
class CacheInputs:
    k: torch.Tensor          # [NL][B][Hkv][Cap][D], workload dtype
    v: torch.Tensor
    length: torch.Tensor     # [NL][B][Hkv] int32
    q_win: torch.Tensor      # [NL][B][Hq][w][D], workload dtype
    reward: np.ndarray       # [B] float32, the step's process reward v in [0, 1]
    seq_len: np.ndarray      # [B] int64, cache length of each sequence
    hitter_dir: torch.Tensor  # [NL][Hkv][D] float32 unit directions


def _rewards(wl: Workload, rng: np.random.Generator, n: int) -> np.ndarray:
    if wl.reward == "uniform":
        v = rng.uniform(0.0, 1.0, size=n)
    elif wl.reward == "beta22":
        v = rng.beta(2.0, 2.0, size=n)
    elif wl.reward == "beta25":
        v = rng.beta(2.0, 5.0, size=n)
    else:
        raise ValueError(wl.reward)
    return v.astype(np.float32)


def make_cache(wl: Workload, device="cpu", capacity: Optional[int] = None,
               n_layers: Optional[int] = None, seq_lens: Optional[Sequence[int]] = None) -> CacheInputs:
    """Draw the pre-compression cache, window queries and rewards of ``wl``.

    ``n_layers`` / ``seq_lens`` shrink the workload for quick tests while keeping
    its per-unit shape.  Rows at or beyond a sequence's length are zero."""
    NL = wl.n_layers if n_layers is None else int(n_layers)
    rng = np.random.default_rng(wl.seed)
    if seq_lens is not None:
        lens = np.asarray(seq_lens, dtype=np.int64)
    elif wl.ragged:
        lo, hi = wl.lengths
        lens = rng.integers(lo, hi + 1, size=wl.batch).astype(np.int64)
    else:
        lens = np.full(wl.batch, int(wl.lengths[0]), dtype=np.int64)
    B = len(lens)
    reward = _rewards(wl, rng, B)
    cap = int(capacity) if capacity is not None else int(lens.max()) + wl.decode_steps
    H, Hq, D, w = wl.n_kv_heads, wl.n_q_heads, wl.head_dim, wl.window
    g = _gen(wl.seed, device)
    k = torch.zeros((NL, B, H, cap, D), dtype=wl.torch_dtype, device=device)
    v = torch.zeros_like(k)
    u = torch.randn((NL, H, D), generator=g, device=device, dtype=torch.float32)
    u = u / torch.linalg.vector_norm(u, dim=-1, keepdim=True)
    for l in range(NL):
        for b in range(B):
            L = int(lens[b])
            kf = torch.randn((H, L, D), generator=g, device=device, dtype=torch.float32)
            vf = torch.randn((H, L, D), generator=g, device=device, dtype=torch.float32)
            n_hit = int(round(wl.hitter_frac * L))
            if n_hit:
                pos = torch.randperm(L, generator=g, device=device)[:n_hit]
                kf[:, pos, :] += wl.hitter_gain * u[l][:, None, :]
                vf[:, pos, :] += wl.hitter_gain * u[l][:, None, :]
            k[l, b, :, :L, :] = kf.to(wl.torch_dtype)
            v[l, b, :, :L, :] = vf.to(wl.torch_dtype)
    q_win = torch.randn((NL, B, Hq, w, D), generator=g, device=device,
                        dtype=torch.float32).to(wl.torch_dtype)
    length = torch.tensor(np.broadcast_to(lens[None, :, None], (NL, B, H)).copy(),
                          dtype=torch.int32, device=device)
    return CacheInputs(k, v, length, q_win, reward, lens, u)


def make_decode_inputs(wl: Workload, cache: CacheInputs, steps: int, seed_offset: int = 0,
                       device="cpu"):
    """Per-step decode query and new K/V rows: lists of ``[NL][B][Hq][D]`` and
    ``[NL][B][Hkv][D]`` tensors.  Each new token is a heavy hitter with
    probability ``hitter_frac`` (per layer and sequence)."""
    NL, B = cache.k.shape[0], cache.k.shape[1]
    H, Hq, D = wl.n_kv_heads, wl.n_q_heads, wl.head_dim
    g = _gen(wl.seed + 7919 + seed_offset, device)
    u = cache.hitter_dir.to(device)
    qs, ks, vs = [], [], []
    for _ in range(steps):
        q = torch.randn((NL, B, Hq, D), generator=g, device=device, dtype=torch.float32)
        kn = torch.randn((NL, B, H, D), generator=g, device=device, dtype=torch.float32)
        vn = torch.randn((NL, B, H, D), generator=g, device=device, dtype=torch.float32)
        hit = (torch.rand((NL, B), generator=g, device=device) < wl.hitter_frac).to(torch.float32)
        bump = wl.hitter_gain * hit[:, :, None, None] * u[:, None, :, :]
        kn += bump
        vn += bump
        qs.append(q.to(wl.torch_dtype))
        ks.append(kn.to(wl.torch_dtype))
        vs.append(vn.to(wl.torch_dtype))
    return qs, ks, vs


def make_logits(rows: int, vocab: int, seed: int, sigma: float = 3.0, device="cpu",
                shape=None) -> torch.Tensor:
    """fp32 logits ~ N(0, sigma^2)."""
    g = _gen(seed, device)
    shp = (rows, vocab) if shape is None else tuple(shape)
    return sigma * torch.randn(shp, generator=g, device=device, dtype=torch.float32)


def make_step_lengths(total: int, mean: float, seed: int) -> np.ndarray:
    """Reasoning-step lengths ~ Geometric(1/mean) until `total` tokens."""
    rng = np.random.default_rng(seed)
    out, t = [], 0
    while t < total:
        n = int(rng.geometric(1.0 / mean))
        n = min(n, total - t)
        out.append(n)
        t += n
    return np.asarray(out, dtype=np.int64)


def make_rewards(kind: str, n: int, batch: int, seed: int) -> np.ndarray:
    """Process rewards [n][batch] ~ U(0,1), Beta(2,2) or Beta(2,5)."""
    rng = np.random.default_rng(seed)
    if kind == "uniform":
        v = rng.uniform(0.0, 1.0, size=(n, batch))
    elif kind == "beta22":
        v = rng.beta(2.0, 2.0, size=(n, batch))
    else:
        v = rng.beta(2.0, 5.0, size=(n, batch))
    return v.astype(np.float32)


def make_reflection_ids(n: int, vocab: int, seed: int) -> np.ndarray:
    """``n`` distinct synthetic reflection-token ids in [0, vocab)."""
    rng = np.random.default_rng(seed)
    return np.sort(rng.choice(vocab, size=n, replace=False)).astype(np.int32)


def make_answer_tokens(batch: int, n: int, vocab: int, seed: int) -> np.ndarray:
    """Uniformly drawn answer token ids ``[batch][n]``."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, vocab, size=(batch, n)).astype(np.int32)


def to_f64(t: torch.Tensor) -> np.ndarray:
    """Exact upcast of an fp32/bf16 tensor to a float64 numpy array."""
    return t.detach().to("cpu").to(torch.float32).numpy().astype(np.float64)


def ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def nbytes_of(dtype: str) -> int:
    return 4 if dtype == "f32" else 2

