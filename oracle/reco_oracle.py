"""CPU oracle for the reward-coordinated compression hot path (fp64, numpy).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or
executes this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may use it.  It shares no code with the HIP
library; both sides only consume the same seeded inputs.

Every function is the plain definition of what the paper's method computes,
written in the paper's order and notation, in float64 unless the paper's step
is itself a float32 operation (the logit penalty).  Library primitives used as
steps: matrix products, ``exp``/``log``, ``np.lexsort`` and ``np.sort``.

Readings taken where the paper is silent (each is also recorded in the
design notes):

* retention: the default reward map is r = clamp(1 - v/2, 0.3, 1); Eq. 1
  (trajectory-relative lambda_i) is available as an alternative policy;
* budget: m = min(L, max(min(w, L), ceil(r * L))) with the product r * L
  taken in IEEE fp64; the most recent min(w, L) tokens are inside the budget;
* Eq. 2 is taken per KV head, summed over the G query heads of its group, with
  logits scaled by 1/sqrt(D) (passed in as ``scale``) and a causal window:
  the window query at position p sees keys 0..p;
* ties in the top-k are broken by the lower (earlier) position;
* decode appends the new token's K/V row before attending to it;
* reflection-penalty bands compare v in float32 exactly as Eq. 3 writes them
  (<=, strict middle band, >=); each distinct reflection id is penalised once;
* answer perplexity uses natural logarithms and the raw logits;
* sampling from softmax(z~ / T) is the Gumbel-max draw argmax(z~ / T + G)
  (T = 0: plain argmax), lowest index on ties, with G from a Philox4x32-10
  stream keyed by (seed, row, offset) -- the paper names no generator.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "retention_from_reward", "retention_eq1", "kept_count", "score_unit", "select_unit",
    "compact_unit", "decode_unit", "penalty_band", "logit_penalty", "answer_ppl",
    "philox4x32_10", "uniform_from_bits", "gumbel_noise", "penalty_sample",
    "layer_retention", "pool_scores",
]


# ---------------------------------------------------------------------------
# Reward -> retention -> budget  (Section 3.2, Eq. 1)
# ---------------------------------------------------------------------------

def retention_from_reward(v: float, lo: float = 0.3, hi: float = 1.0) -> float:
    """Default reward-to-retention map r(v) = clamp(1 - v/2, lo, hi) in fp64.

    Higher process reward means a more reliable state, hence harder pruning
    (Section 3.2, reward-driven retention)."""
    r = 1.0 - 0.5 * float(v)
    return min(hi, max(lo, r))


def retention_eq1(v_hist: Sequence[float], lam: float = 0.25, delta: float = 0.1) -> float:
    """Eq. 1: lambda_i = lambda - delta * (v_i - mean(v)) / (max(v) - min(v)).

    ``v_hist`` holds the step rewards of the trajectory so far, the latest step
    last (it is included in the statistics).  When all rewards are equal the
    adjustment is undefined; the reading taken is lambda_i = lambda."""
    v = np.asarray(v_hist, dtype=np.float64)
    if v.size == 0:
        raise ValueError("empty reward history")
    vmax, vmin = float(v.max()), float(v.min())
    if vmax == vmin:
        return float(lam)
    return float(lam - delta * (float(v[-1]) - float(v.mean())) / (vmax - vmin))


def kept_count(L: int, w: int, r: float) -> int:
    """Budget m_i = lambda_i * L of Section 3.2, rounded up, with the window of
    the w most recent tokens always kept (and counted inside the budget)."""
    if not (0.0 < r <= 1.0):
        raise ValueError("retention must lie in (0, 1]")
    w_eff = min(int(w), int(L))
    return min(int(L), max(w_eff, math.ceil(float(r) * float(L))))


def layer_retention(r: float, layer: int, n_layers: int, spread: float) -> float:
    """Per-layer budgets, a policy variant on the same kernels (the pyramid
    idea the paper cites among classical eviction methods, Section 1): the
    retention falls linearly with depth from r(1 + spread) at layer 0 to
    r(1 - spread) at the last layer, so its mean over layers is r, and is
    capped at 1 (a cap lowers the mean).  spread = 0 is the paper's single
    retention level; 0 <= spread < 1."""
    if not (0.0 <= spread < 1.0):
        raise ValueError("spread must lie in [0, 1)")
    if n_layers == 1:
        return min(1.0, float(r))
    t = float(layer) / float(n_layers - 1)
    return min(1.0, float(r) * (1.0 + float(spread) * (1.0 - 2.0 * t)))


# ---------------------------------------------------------------------------
# Attention-guided importance  (Section 3.2, Eq. 2)
# ---------------------------------------------------------------------------

def score_unit(K: np.ndarray, Qwin: np.ndarray, scale: float, causal: bool = True) -> np.ndarray:
    """Eq. 2 for one (layer, sequence, kv head):
    s_j = sum over window queries t of softmax_j(scale * q_t . k_j).

    K    : [L][D] cached keys of this KV head (fp64).
    Qwin : [G][w][D] window queries of the G query heads that share this KV
           head; row t of the window is the query of absolute position
           L - w + t (rows with a negative position do not exist).
    Returns s : [L] fp64, one score per cached key (window keys included)."""
    K = np.asarray(K, dtype=np.float64)
    Qwin = np.asarray(Qwin, dtype=np.float64)
    L = K.shape[0]
    G, w, D = Qwin.shape
    w_eff = min(w, L)
    s = np.zeros(L, dtype=np.float64)
    if L == 0:
        return s
    rows = Qwin[:, w - w_eff:, :].reshape(G * w_eff, D)        # [G*w_eff][D]
    pos = np.tile(np.arange(L - w_eff, L), G)                    # absolute position of each row
    logits = scale * (rows @ K.T)                                # [G*w_eff][L]
    if causal:
        logits = np.where(np.arange(L)[None, :] <= pos[:, None], logits, -np.inf)
    logits = logits - logits.max(axis=1, keepdims=True)
    e = np.exp(logits)
    p = e / e.sum(axis=1, keepdims=True)                         # softmax over keys, per row
    s += p.sum(axis=0)                                           # sum over the window
    return s


# ---------------------------------------------------------------------------
# Selection and compaction  (Section 3.2, attention-guided selection)
# ---------------------------------------------------------------------------

def select_unit(s: np.ndarray, L: int, w: int, r: float) -> np.ndarray:
    """Keep the m highest-scoring tokens, the w most recent always kept.

    The window [L - w_eff, L) is forced; the remaining k = m - w_eff slots go
    to the prefix positions with the largest score, ties to the earlier
    position.  Returns the kept positions in ascending order (length m)."""
    L = int(L)
    w_eff = min(int(w), L)
    m = kept_count(L, w, r)
    k = m - w_eff
    P = L - w_eff
    prefix = np.asarray(s, dtype=np.float64)[:P]
    order = np.lexsort((np.arange(P), -prefix))                  # score desc, then position asc
    kept = np.sort(order[:k])
    return np.concatenate([kept, np.arange(P, L)]).astype(np.int64)


def pool_scores(s: np.ndarray, L: int, w: int, kernel: int, mode: str) -> np.ndarray:
    """Score pooling before the top-k, a policy variant on the same kernels
    (the clustering idea of SnapKV, cited in Section 1): each prefix position
    j < P = L - min(w, L) takes the max ("max") or the mean ("mean") of s
    over the prefix positions i with |i - j| <= kernel // 2; window positions
    keep their own score (the window is always kept).  kernel is odd."""
    L = int(L)
    P = L - min(int(w), L)
    h = int(kernel) // 2
    s = np.asarray(s, dtype=np.float64)
    out = s[:L].copy()
    if P == 0:
        return out
    padded = np.concatenate([np.full(h, np.nan), s[:P], np.full(h, np.nan)])
    win = np.lib.stride_tricks.sliding_window_view(padded, 2 * h + 1)    # [P][kernel], NaN outside the prefix
    out[:P] = np.nanmax(win, axis=1) if mode == "max" else np.nanmean(win, axis=1)
    return out


def compact_unit(K: np.ndarray, V: np.ndarray, idx: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Retained cache: K'[p] = K[idx[p]], V'[p] = V[idx[p]] for p < m."""
    idx = np.asarray(idx, dtype=np.int64)
    return K[idx].copy(), V[idx].copy()


# ---------------------------------------------------------------------------
# Decode attention over the retained cache (per-token attention cost, Section 1)
# ---------------------------------------------------------------------------

def decode_unit(K: np.ndarray, V: np.ndarray, n: int, Q: np.ndarray, scale: float,
                k_new: Optional[np.ndarray] = None, v_new: Optional[np.ndarray] = None):
    """Softmax attention of the G query heads of one KV group over its cache.

    K, V : [>=n][D]; the first n rows are the retained cache.
    Q    : [G][D] queries of the group's query heads.
    k_new, v_new : [D] the new token's key/value, appended as row n before
                   attending (the generated token attends to itself).
    Returns (out [G][D], lse [G]) with lse the natural log-sum-exp of the
    scaled logits."""
    K = np.asarray(K, dtype=np.float64)[:n]
    V = np.asarray(V, dtype=np.float64)[:n]
    if k_new is not None:
        K = np.vstack([K, np.asarray(k_new, dtype=np.float64)[None, :]])
        V = np.vstack([V, np.asarray(v_new, dtype=np.float64)[None, :]])
    Q = np.asarray(Q, dtype=np.float64)
    if K.shape[0] == 0:
        return np.zeros((Q.shape[0], Q.shape[1])), np.full(Q.shape[0], -np.inf)
    a = scale * (Q @ K.T)                                        # [G][n]
    M = a.max(axis=1, keepdims=True)
    e = np.exp(a - M)
    Z = e.sum(axis=1, keepdims=True)
    out = (e @ V) / Z
    lse = (M + np.log(Z))[:, 0]
    return out, lse


# ---------------------------------------------------------------------------
# Reward-banded reflection penalty  (Section 3.3, Eq. 3 and Eq. 4)
# ---------------------------------------------------------------------------

def penalty_band(v, tau_lo, tau_hi, beta_lo, beta_mid, beta_hi) -> np.float32:
    """Eq. 3 band, with the comparisons taken in float32 as written."""
    v = np.float32(v)
    if v <= np.float32(tau_lo):
        return np.float32(beta_lo)
    if v >= np.float32(tau_hi):
        return np.float32(beta_hi)
    return np.float32(beta_mid)


def logit_penalty(z: np.ndarray, refl_ids: Sequence[int], reward: Sequence[float],
                  tau_lo: float, tau_hi: float, beta_lo: float, beta_mid: float,
                  beta_hi: float) -> np.ndarray:
    """Eq. 4: z~(u) = z(u) - beta_i for every reflection token u in R (a set),
    all other logits unchanged.  Works on a float32 copy of ``z`` [rows][vocab];
    row b uses reward[b]."""
    out = np.array(z, dtype=np.float32, copy=True)
    ids = sorted(set(int(u) for u in refl_ids))
    for b in range(out.shape[0]):
        beta = penalty_band(reward[b], tau_lo, tau_hi, beta_lo, beta_mid, beta_hi)
        for u in ids:
            out[b, u] = np.float32(out[b, u] - beta)
    return out


# ---------------------------------------------------------------------------
# Answer perplexity and the stopping rule  (Section 3.3, Eq. 5 and Eq. 6)
# ---------------------------------------------------------------------------

def answer_ppl(logits: np.ndarray, tokens: np.ndarray, tau_p: float):
    """Eq. 5: PPL(a) = exp(-(1/n) sum_t log p(x_t | x_<t)), where p is the
    softmax of the logit row at step t; Eq. 6: stop when PPL <= tau_p.

    logits : [B][n][V] (any float type, taken in fp64); tokens : [B][n].
    Returns (ppl [B] fp64, stop [B] bool)."""
    z = np.asarray(logits, dtype=np.float64)
    x = np.asarray(tokens, dtype=np.int64)
    B, n, _ = z.shape
    M = z.max(axis=2, keepdims=True)
    lse = (M + np.log(np.exp(z - M).sum(axis=2, keepdims=True)))[:, :, 0]     # [B][n]
    logp = np.take_along_axis(z, x[:, :, None], axis=2)[:, :, 0] - lse
    nll = -logp.mean(axis=1)
    ppl = np.exp(nll)
    stop = ppl <= float(np.float32(tau_p))
    return ppl, stop


# ---------------------------------------------------------------------------
# Whole-cache drivers: plain loops over (layer, sequence, kv head) units.
# Query head hq belongs to KV head hq // G (G = n_q_heads / n_kv_heads).
# ---------------------------------------------------------------------------

def score_cache(K: np.ndarray, lens: np.ndarray, Qwin: np.ndarray, scale: float,
                causal: bool = True, units=None) -> np.ndarray:
    """Eq. 2 over a cache K [NL][B][H][Cap][D] with lengths lens [NL][B][H] and
    window queries Qwin [NL][B][Hq][w][D].  Returns s [NL][B][H][Cap] (zero at
    and beyond each unit's length).  ``units`` optionally restricts the work
    to an iterable of (layer, seq, head) triples."""
    NL, B, H, Cap, D = K.shape
    G = Qwin.shape[2] // H
    s = np.zeros((NL, B, H, Cap), dtype=np.float64)
    it = units if units is not None else ((l, b, h) for l in range(NL) for b in range(B) for h in range(H))
    for (l, b, h) in it:
        L = int(lens[l, b, h])
        s[l, b, h, :L] = score_unit(K[l, b, h, :L], Qwin[l, b, h * G:(h + 1) * G], scale, causal)
    return s


def compress_cache(K: np.ndarray, V: np.ndarray, lens: np.ndarray, Qwin: np.ndarray,
                   retention: Sequence[float], w: int, scale: float, causal: bool = True):
    """Score, select and compact every unit (retention r is per sequence,
    ``retention[b]``, or per layer and sequence, ``retention[l][b]``).

    Returns (s, idx, K2, V2, lens2): scores, the kept index list of every unit
    (dict keyed by (layer, seq, head)), the compacted caches (rows >= m keep
    their old contents) and the new lengths."""
    s = score_cache(K, lens, Qwin, scale, causal)
    K2, V2, lens2 = K.copy(), V.copy(), lens.copy()
    idx = {}
    NL, B, H = lens.shape
    for l in range(NL):
        for b in range(B):
            for h in range(H):
                L = int(lens[l, b, h])
                r = retention[b] if np.ndim(retention) == 1 else retention[l][b]
                sel = select_unit(s[l, b, h], L, w, float(r))
                idx[(l, b, h)] = sel
                kk, vv = compact_unit(K[l, b, h], V[l, b, h], sel)
                K2[l, b, h, :len(sel)] = kk
                V2[l, b, h, :len(sel)] = vv
                lens2[l, b, h] = len(sel)
    return s, idx, K2, V2, lens2


def decode_cache(K: np.ndarray, V: np.ndarray, lens: np.ndarray, Q: np.ndarray, scale: float,
                 k_new: Optional[np.ndarray] = None, v_new: Optional[np.ndarray] = None,
                 units=None):
    """One decode step over every unit.  Q [NL][B][Hq][D]; k_new, v_new
    [NL][B][H][D] or None.  Returns (out [NL][B][Hq][D], lse [NL][B][Hq]).
    When appending, the new rows are written into K, V (in place) and lens is
    incremented, as the cache of a generating model would be."""
    NL, B, H, Cap, D = K.shape
    Hq = Q.shape[2]
    G = Hq // H
    out = np.zeros((NL, B, Hq, D), dtype=np.float64)
    lse = np.zeros((NL, B, Hq), dtype=np.float64)
    it = units if units is not None else [(l, b, h) for l in range(NL) for b in range(B) for h in range(H)]
    for (l, b, h) in it:
        n = int(lens[l, b, h])
        kn = None if k_new is None else k_new[l, b, h]
        vn = None if v_new is None else v_new[l, b, h]
        o, z = decode_unit(K[l, b, h], V[l, b, h], n, Q[l, b, h * G:(h + 1) * G], scale, kn, vn)
        out[l, b, h * G:(h + 1) * G] = o
        lse[l, b, h * G:(h + 1) * G] = z
        if kn is not None:
            K[l, b, h, n] = kn
            V[l, b, h, n] = vn
            lens[l, b, h] = n + 1
    return out, lse


# ---------------------------------------------------------------------------
# Penalised sampling (Section 3.3: sample from softmax of the penalised logits)
# ---------------------------------------------------------------------------

# Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy
# as 1, 2, 3", SC 2011): multipliers and Weyl key increments of the paper.
_PHILOX_M0, _PHILOX_M1 = 0xD2511F53, 0xCD9E8D57
_PHILOX_W0, _PHILOX_W1 = 0x9E3779B9, 0xBB67AE85


def philox4x32_10(counter, key):
    """Philox4x32 with 10 rounds.  counter: four uint32 arrays (broadcast
    together), key: two uint32 scalars.  Returns four uint32 arrays."""
    mask = np.uint64(0xFFFFFFFF)
    c = [np.asarray(x, dtype=np.uint64) for x in counter]
    k0, k1 = np.uint64(key[0]), np.uint64(key[1])
    for rnd in range(10):
        p0 = np.uint64(_PHILOX_M0) * c[0]
        p1 = np.uint64(_PHILOX_M1) * c[2]
        hi0, lo0 = p0 >> np.uint64(32), p0 & mask
        hi1, lo1 = p1 >> np.uint64(32), p1 & mask
        c = [hi1 ^ c[1] ^ k0, lo1, hi0 ^ c[3] ^ k1, lo0]
        if rnd < 9:
            k0 = (k0 + np.uint64(_PHILOX_W0)) & mask
            k1 = (k1 + np.uint64(_PHILOX_W1)) & mask
    return [x.astype(np.uint32) for x in c]


def uniform_from_bits(x: np.ndarray) -> np.ndarray:
    """Open-interval uniform from 32 random bits, float32: the top 23 bits
    pick one of 2^23 equal cells of (0, 1) and U is the cell's midpoint,
    (k + 1/2) * 2^-23 with k = x >> 9.  Every midpoint is an exact float32
    (2k + 1 < 2^24), so U never rounds to 0 or 1 and U(x) + U(~x) = 1."""
    k = (np.asarray(x, dtype=np.uint32) >> np.uint32(9)).astype(np.float32)
    return (k * np.float32(2.0 ** -23) + np.float32(2.0 ** -24)).astype(np.float32)


def gumbel_noise(row: int, vocab: int, seed: int, offset: int) -> np.ndarray:
    """Gumbel(0,1) noise of one logit row, float32: G_j = -log(-log(U_j)),
    U_j = uniform_from_bits(x_j), x_j the (j % 4)-th output of Philox on
    counter (j / 4, row, offset low, offset high), key (seed low, seed high)."""
    j = np.arange(vocab, dtype=np.uint64)
    blk = j // np.uint64(4)
    outs = philox4x32_10([blk, np.full_like(blk, row), np.full_like(blk, offset & 0xFFFFFFFF),
                          np.full_like(blk, (offset >> 32) & 0xFFFFFFFF)],
                         (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF))
    x = np.choose((j % np.uint64(4)).astype(np.int64), outs).astype(np.uint32)
    u = uniform_from_bits(x)
    return (-np.log(-np.log(u))).astype(np.float32)


def penalty_sample(z: np.ndarray, refl_ids, reward, tau_lo, tau_hi, beta_lo, beta_mid, beta_hi,
                   temperature: float, seed: int, offset: int):
    """Eq. 3-4 on every row, then the next token of each row from
    softmax(z~ / T): argmax of z~ (T = 0, lowest index on ties) or the
    Gumbel-max draw argmax(z~ / T + G).  Returns (penalised float32 rows,
    tokens int64, the float32 values the argmax was taken over)."""
    zp = logit_penalty(z, refl_ids, reward, tau_lo, tau_hi, beta_lo, beta_mid, beta_hi)
    rows, vocab = zp.shape
    vals = np.empty_like(zp)
    for b in range(rows):
        if temperature == 0:
            vals[b] = zp[b]
        else:
            vals[b] = (zp[b] / np.float32(temperature)).astype(np.float32) + gumbel_noise(b, vocab, seed, offset)
    tokens = np.argmax(vals, axis=1)           # first maximum: lowest index on ties
    return zp, tokens.astype(np.int64), vals
