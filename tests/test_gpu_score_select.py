"""GPU parity of reco_score (Eq. 2) and reco_select_compact against the oracle."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import WORST_NEAR_THETA, SCORE_RTOL, assert_theta_precision, f64, kept_sets_match, upload
from paper_2608_04771_amd import binding as B
from paper_2608_04771_amd import inputs as I

pytestmark = pytest.mark.gpu


def _score_check(cache_in, q_win, w, causal=True, D=None):
    cache = upload(cache_in) if isinstance(cache_in, I.CacheInputs) else cache_in
    D = cache.shape[-1]
    dev_err = torch.zeros(1, dtype=torch.int32, device="cuda")
    s = B.reco_score(cache, q_win.cuda(), w, causal=causal, dev_err=dev_err)
    torch.cuda.synchronize()
    assert dev_err.item() == 0
    K = f64(cache.k)
    lens = cache.length.cpu().numpy()
    ref = oracle.score_cache(K, lens, f64(q_win), 1 / np.sqrt(D), causal)
    g = s.cpu().numpy().astype(np.float64)
    worst = 0.0
    for u in np.ndindex(*lens.shape):
        L = int(lens[u])
        if L == 0:
            continue
        rel = np.abs(g[u][:L] - ref[u][:L]) / np.maximum(ref[u][:L], 1e-30)
        big = ref[u][:L] > 1e-20
        worst = max(worst, float(rel[big].max()) if big.any() else 0.0)
        G = q_win.shape[2] // lens.shape[2]
        assert abs(g[u][:L].sum() - G * min(w, L)) <= 1e-4 * G * min(w, L)     # mass invariant
        for r in (0.5, 0.75, 0.9):                                             # the workloads' retention range
            assert_theta_precision(g[u], ref[u], L, w, r, f"unit {u} r={r}")
    assert worst <= SCORE_RTOL, f"score rel err {worst:.3e}"
    return s, ref, worst


def test_score_tiny_workload():
    wl = I.WORKLOADS["tiny"]
    ci = I.make_cache(wl)
    _, _, worst = _score_check(ci, ci.q_win, wl.window)
    print(f"tiny score max rel err {worst:.3e}")


@pytest.mark.parametrize("dtype,D,G,w", [("bf16", 128, 7, 64), ("bf16", 128, 5, 32), ("f32", 128, 4, 16),
                                         ("bf16", 64, 1, 8), ("bf16", 128, 8, 100),
                                         ("bf16", 64, 16, 256),                  # G*w = 4096 rows, the limit
                                         ("f32", 64, 16, 256), ("f32", 128, 8, 64)])
@pytest.mark.parametrize("causal", [True, False])
def test_score_ragged(dtype, D, G, w, causal):
    H, NL, Bsz = 2, 2, 2
    Cap = 1300
    lens = [1300, 1, 7, 64, 65, 513, 1024, 1025]
    gen = torch.Generator().manual_seed(D + G + w)
    td = torch.float32 if dtype == "f32" else torch.bfloat16
    k = torch.randn((NL, Bsz, H, Cap, D), generator=gen).to(td)
    v = torch.zeros_like(k)
    ln = torch.tensor(lens, dtype=torch.int32).reshape(NL, Bsz, H)
    q = torch.randn((NL, Bsz, H * G, w, D), generator=gen).to(td)
    cache = B.KVCache(k.cuda(), v.cuda(), ln.cuda())
    _, _, worst = _score_check(cache, q, w, causal)
    print(f"{dtype} D={D} G={G} w={w} causal={causal} max rel err {worst:.3e}; worst near theta so far "
          f"{WORST_NEAR_THETA['rel']:.3e} ({WORST_NEAR_THETA['where']})")


def test_select_compact_tiny_end_to_end():
    """GPU score -> GPU select/compact, compared with the oracle's selection on
    the oracle's own scores (ties excused) and bit-exact gathered rows."""
    wl = I.WORKLOADS["tiny"]
    ci = I.make_cache(wl)
    cache = upload(ci)
    s = B.reco_score(cache, ci.q_win.cuda(), wl.window)
    r = oracle.retention_from_reward(float(ci.reward[0]))
    ret = torch.tensor([B.reco_retention_from_reward(float(ci.reward[0]))], dtype=torch.float64, device="cuda")
    assert ret.item() == r
    kept = torch.full((1, 1, wl.n_kv_heads, cache.shape[3]), -1, dtype=torch.int32, device="cuda")
    k0, v0 = cache.k.clone(), cache.v.clone()
    dev_err = torch.zeros(1, dtype=torch.int32, device="cuda")
    B.reco_select_compact(cache, s, ret, wl.window, kept_idx=kept, dev_err=dev_err)
    torch.cuda.synchronize()
    assert dev_err.item() == 0
    s_or = oracle.score_cache(f64(ci.k), ci.length.numpy(), f64(ci.q_win), 1 / np.sqrt(wl.head_dim))
    L = int(ci.seq_len[0])
    m = oracle.kept_count(L, wl.window, r)
    kk = kept.cpu().numpy()
    for h in range(wl.n_kv_heads):
        ok, msg = kept_sets_match(kk[0, 0, h], s_or[0, 0, h], L, wl.window, r)
        assert ok, msg
        # the select kernel alone is exact on the GPU's own scores
        exact = oracle.select_unit(s.cpu().numpy()[0, 0, h].astype(np.float64), L, wl.window, r)
        assert (kk[0, 0, h, :m] == exact).all()
        idx = torch.from_numpy(kk[0, 0, h, :m].astype(np.int64)).cuda()
        assert torch.equal(cache.k[0, 0, h, :m], k0[0, 0, h][idx])
        assert torch.equal(cache.v[0, 0, h, :m], v0[0, 0, h][idx])
    assert (cache.length.cpu().numpy() == m).all()


def _pattern_scores(kind, L, rng):
    j = np.arange(L, dtype=np.float64)
    if kind == "keep_first":
        return (L - j) / L
    if kind == "keep_last":
        return (j + 1) / L
    if kind == "every_other":
        return np.where(j % 2 == 0, 2.0, 1.0) + j * 1e-9
    if kind == "single_gap":
        s = np.ones(L)
        s[L // 3] = 0.0
        return s
    if kind == "all_equal":
        return np.full(L, 0.25)
    if kind == "random":
        return rng.random(L)
    if kind == "few_levels":
        return rng.integers(0, 5, L) / 4.0
    raise ValueError(kind)


@pytest.mark.parametrize("kind", ["keep_first", "keep_last", "every_other", "single_gap", "all_equal",
                                  "random", "few_levels"])
@pytest.mark.parametrize("dtype,D", [("bf16", 128), ("f32", 64)])
def test_select_compact_patterns(kind, dtype, D):
    """Adversarial selection patterns on given scores: indices must equal the
    oracle exactly (same fp32 scores) and rows must move bit-exactly."""
    rng = np.random.default_rng(7)
    NL, Bsz, H, Cap, w = 1, 3, 2, 5000, 32
    lens = [5000, 4097, 1000, 33, 32, 2]
    ret_np = np.array([0.5, 0.3, 0.77], dtype=np.float64)
    if kind == "single_gap":
        ret_np = np.array([1 - 1 / 5000, 0.999, 0.999])
    td = torch.float32 if dtype == "f32" else torch.bfloat16
    gen = torch.Generator().manual_seed(11)
    k = torch.randn((NL, Bsz, H, Cap, D), generator=gen).to(td)
    v = torch.randn((NL, Bsz, H, Cap, D), generator=gen).to(td)
    ln = torch.tensor(lens, dtype=torch.int32).reshape(NL, Bsz, H)
    sc = np.zeros((NL, Bsz, H, Cap), dtype=np.float32)
    for u in np.ndindex(NL, Bsz, H):
        L = int(ln[u])
        sc[u][:L] = _pattern_scores(kind, L, rng).astype(np.float32)
    cache = B.KVCache(k.cuda(), v.cuda(), ln.cuda())
    kept = torch.full((NL, Bsz, H, Cap), -1, dtype=torch.int32, device="cuda")
    dev_err = torch.zeros(1, dtype=torch.int32, device="cuda")
    B.reco_select_compact(cache, torch.from_numpy(sc).cuda(), torch.from_numpy(ret_np).cuda(), w,
                          kept_idx=kept, dev_err=dev_err)
    torch.cuda.synchronize()
    assert dev_err.item() == 0
    kk = kept.cpu().numpy()
    kc, vc, lc = cache.k.cpu(), cache.v.cpu(), cache.length.cpu().numpy()
    for u in np.ndindex(NL, Bsz, H):
        L = int(ln[u])
        r = float(ret_np[u[1]])
        ref = oracle.select_unit(sc[u].astype(np.float64), L, w, r)
        m = len(ref)
        assert lc[u] == m
        assert (kk[u][:m] == ref).all(), (kind, u)
        idx = torch.from_numpy(ref)
        assert torch.equal(kc[u][:m], k[u][idx]) and torch.equal(vc[u][:m], v[u][idx])


def test_select_rejects_bad_retention_and_scores():
    NL, Bsz, H, Cap, D, w = 1, 2, 1, 256, 128, 8
    k = torch.randn((NL, Bsz, H, Cap, D)).to(torch.bfloat16)
    v = torch.randn((NL, Bsz, H, Cap, D)).to(torch.bfloat16)
    ln = torch.full((NL, Bsz, H), 200, dtype=torch.int32)
    sc = torch.rand((NL, Bsz, H, Cap))
    cache = B.KVCache(k.cuda(), v.cuda(), ln.cuda())
    dev_err = torch.zeros(1, dtype=torch.int32, device="cuda")
    B.reco_select_compact(cache, sc.cuda(), torch.tensor([0.0, 0.5], dtype=torch.float64, device="cuda"), w,
                          dev_err=dev_err)
    torch.cuda.synchronize()
    assert dev_err.item() == 2
    assert cache.length.cpu().tolist() == [[[200], [100]]]                 # seq 0 untouched
    assert torch.equal(cache.k.cpu()[0, 0], k[0, 0])
    sc[0, 1, 0, 5] = float("nan")
    dev_err.zero_()
    B.reco_select_compact(cache, sc.cuda(), torch.tensor([0.5, 0.5], dtype=torch.float64, device="cuda"), w,
                          dev_err=dev_err)
    torch.cuda.synchronize()
    assert dev_err.item() == 3
    assert cache.length.cpu().tolist() == [[[100], [100]]]                 # seq 1 (NaN) untouched
