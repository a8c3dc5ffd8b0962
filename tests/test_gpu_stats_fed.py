"""GPU parity of scoring fed with the decode statistics of the window tokens
(one pass over K): decode's (max, sum) pairs agree with its lse and with the
oracle's logit maxima, and after w decode steps with no compression in
between, reco_score with those statistics matches the oracle's Eq. 2 and the
two-pass scores, and selects the same keys (ties excused)."""
import math

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import SCORE_RTOL, assert_theta_precision, f64, kept_sets_match
from paper_2608_04771_amd import binding as B
from paper_2608_04771_amd import inputs as I

pytestmark = pytest.mark.gpu

LOG2E = 1.4426950408889634


def _decode_window(cache, Hq, w, n_tokens, seed, td):
    """Decode n_tokens (appending each); returns the queries [NL][B][Hq][n][D]
    and the row statistics [NL][B][Hq][n][2] of every token."""
    NL, Bsz, H, Cap, D = cache.shape
    g = torch.Generator().manual_seed(seed)
    qs, stats = [], []
    for _ in range(n_tokens):
        q = torch.randn((NL, Bsz, Hq, D), generator=g).to(td).cuda()
        kn = torch.randn((NL, Bsz, H, D), generator=g).to(td).cuda()
        vn = torch.randn((NL, Bsz, H, D), generator=g).to(td).cuda()
        st = torch.empty((NL, Bsz, Hq, 2), dtype=torch.float32, device="cuda")
        B.reco_decode_attn(cache, q, kn, vn, row_stats=st)
        qs.append(q)
        stats.append(st)
    return torch.stack(qs, dim=3).contiguous(), torch.stack(stats, dim=3).contiguous()


@pytest.mark.parametrize("dtype,D", [("f32", 64), ("bf16", 128)])
def test_decode_row_stats_are_the_softmax_normalisers(dtype, D):
    td = torch.float32 if dtype == "f32" else torch.bfloat16
    NL, Bsz, H, Hq, Cap = 2, 2, 2, 8, 3000
    lens = [[2999, 100], [0, 1500]]
    g = torch.Generator().manual_seed(4)
    k = torch.randn((NL, Bsz, H, Cap, D), generator=g).to(td)
    v = torch.randn((NL, Bsz, H, Cap, D), generator=g).to(td)
    ln = torch.tensor([[[lens[b][h] for h in range(H)] for b in range(Bsz)]] * NL, dtype=torch.int32)
    cache = B.KVCache(k.cuda(), v.cuda(), ln.cuda())
    q = torch.randn((NL, Bsz, Hq, D), generator=g).to(td)
    st = torch.empty((NL, Bsz, Hq, 2), dtype=torch.float32, device="cuda")
    _, lse = B.reco_decode_attn(cache, q.cuda(), row_stats=st)
    torch.cuda.synchronize()
    st, lse = st.cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)
    K, Q = f64(k), f64(q)
    scale = 1 / math.sqrt(D)
    G = Hq // H
    for l in range(NL):
        for b in range(Bsz):
            for hq in range(Hq):
                n = int(ln[l, b, hq // G])
                M, Z = st[l, b, hq]
                if n == 0:
                    assert M == -np.inf and Z == 0
                    continue
                x = scale * LOG2E * (K[l, b, hq // G, :n] @ Q[l, b, hq])
                assert abs(M - x.max()) <= 1e-5 * max(1.0, abs(x.max()))
                assert Z == pytest.approx(np.exp2(x - x.max()).sum(), rel=1e-5)
                assert (M + math.log2(Z)) * math.log(2) == pytest.approx(lse[l, b, hq], abs=1e-5)


@pytest.mark.parametrize("dtype,D,G,w,prompt", [("f32", 64, 4, 16, 700), ("bf16", 128, 7, 32, 2500),
                                                ("bf16", 64, 2, 16, 0)])
def test_stats_fed_score_matches_oracle(dtype, D, G, w, prompt):
    """The last case starts from an empty cache and decodes fewer than w
    tokens, so the leading window rows have no position (absent rows)."""
    td = torch.float32 if dtype == "f32" else torch.bfloat16
    NL, Bsz, H = 2, 2, 2
    Hq = G * H
    n_tok = w if prompt >= w else 6
    Cap = max(prompt + n_tok, w) + 8                     # w <= capacity
    g = torch.Generator().manual_seed(9)
    k = torch.zeros((NL, Bsz, H, Cap, D), dtype=td)
    v = torch.zeros_like(k)
    k[:, :, :, :prompt] = torch.randn((NL, Bsz, H, prompt, D), generator=g).to(td)
    v[:, :, :, :prompt] = torch.randn((NL, Bsz, H, prompt, D), generator=g).to(td)
    ln = torch.full((NL, Bsz, H), prompt, dtype=torch.int32)
    cache = B.KVCache(k.cuda(), v.cuda(), ln.cuda())
    qs, stats = _decode_window(cache, Hq, w, n_tok, seed=10, td=td)
    if n_tok < w:                                          # rows of positions < 0 exist in the buffers only
        pad = w - n_tok
        qs = torch.cat([torch.zeros_like(qs[:, :, :, :1]).expand(-1, -1, -1, pad, -1), qs], dim=3).contiguous()
        stats = torch.cat([torch.zeros_like(stats[:, :, :, :1]).expand(-1, -1, -1, pad, -1), stats], dim=3).contiguous()
    s_fed = B.reco_score(cache, qs, w, row_stats=stats)
    s_two = B.reco_score(cache, qs, w)
    torch.cuda.synchronize()
    Kc = f64(cache.k)
    lens = cache.length.cpu().numpy()
    assert (lens == prompt + n_tok).all()
    s_or = oracle.score_cache(Kc, lens, f64(qs), 1 / math.sqrt(D))
    a, b2 = s_fed.cpu().numpy().astype(np.float64), s_two.cpu().numpy().astype(np.float64)
    for u in np.ndindex(*lens.shape):
        L = int(lens[u])
        ref = s_or[u][:L]
        big = ref > 1e-20
        rel = np.abs(a[u][:L] - ref)[big] / ref[big]
        assert rel.max() <= SCORE_RTOL, (u, rel.max())
        assert np.abs(a[u][:L] - b2[u][:L]).max() <= 2 * SCORE_RTOL * max(1.0, ref.max())
        assert abs(a[u][:L].sum() - G * min(w, L)) <= 1e-4 * G * min(w, L)
        for r in (0.3, 0.6):
            kept = oracle.select_unit(a[u], L, w, r)                       # GPU scores, oracle's selection rule
            ok, msg = kept_sets_match(kept, ref, L, w, r)
            assert ok, (u, r, msg)
            assert_theta_precision(a[u], ref, L, w, r, f"one-pass unit {u} r={r}")
