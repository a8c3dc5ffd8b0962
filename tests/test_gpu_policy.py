"""GPU parity of the policy variants on the same kernels: score pooling
(reco_pool_scores) and per-layer budgets (reco_select_compact with a
[layer][sequence] retention), alone and behind the real scoring kernel."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import f64, kept_sets_match
from paper_2608_04771_amd import binding as B
from paper_2608_04771_amd import inputs as I

pytestmark = pytest.mark.gpu


def _cache(lens, Cap, D=64, NL=None, dtype=torch.float32, seed=3):
    lens = np.asarray(lens)
    g = torch.Generator().manual_seed(seed)
    shp = tuple(lens.shape) + (Cap, D)
    k = torch.randn(shp, generator=g).to(dtype)
    v = torch.randn(shp, generator=g).to(dtype)
    ln = torch.from_numpy(lens.astype(np.int32))
    return B.KVCache(k.cuda(), v.cuda(), ln.cuda()), k, v


@pytest.mark.parametrize("mode", ["max", "mean"])
@pytest.mark.parametrize("kernel", [1, 3, 7, 65])
def test_pool_matches_oracle(mode, kernel):
    """Ragged units (empty, shorter than the window, chunk edges, full
    capacity); maxima bit-exact, means within one fp32 rounding."""
    Cap, w = 6000, 32
    lens = np.array([[[6000, 0, 20, 33], [2048, 2049, 4097, 32]], [[1, 5000, 2081, 4000], [6000, 3, 64, 2047]]])
    cache, _, _ = _cache(lens, Cap)
    rng = np.random.default_rng(kernel)
    sc = rng.exponential(size=lens.shape + (Cap,)).astype(np.float32)
    sc[0, 0, 0, 100:200] = 0.0                                            # flat stretch and a spike
    sc[0, 0, 0, 150] = 50.0
    pooled = torch.full(sc.shape, float("nan"), dtype=torch.float32, device="cuda")
    dev_err = torch.zeros(1, dtype=torch.int32, device="cuda")
    B.reco_pool_scores(cache, torch.from_numpy(sc).cuda(), w, kernel, mode, pooled=pooled, dev_err=dev_err)
    torch.cuda.synchronize()
    assert dev_err.item() == 0
    got = pooled.cpu().numpy()
    for u in np.ndindex(*lens.shape):
        L = int(lens[u])
        ref = oracle.pool_scores(sc[u].astype(np.float64), L, w, kernel, mode)
        if mode == "max":
            assert got[u][:L].tobytes() == ref.astype(np.float32).tobytes(), u
        else:
            np.testing.assert_allclose(got[u][:L], ref, rtol=2.0 ** -24, atol=0, err_msg=str(u))
        assert np.isnan(got[u][L:]).all(), u                               # beyond len: not written


def test_per_layer_budgets_select_exactly():
    NL, Bsz, H, Cap, w = 4, 2, 2, 3000, 16
    lens = np.zeros((NL, Bsz, H), dtype=np.int64)
    lens[:] = [[3000, 2500], [17, 1200]]
    cache, k, v = _cache(lens, Cap, D=128, dtype=torch.bfloat16)
    sc = np.random.default_rng(0).random((NL, Bsz, H, Cap)).astype(np.float32)
    base = [0.5807587504386902, 0.3]
    ret = np.array([[oracle.layer_retention(r, l, NL, 0.6) for r in base] for l in range(NL)])
    ret_dev = torch.tensor([[B.reco_layer_retention(r, l, NL, 0.6) for r in base] for l in range(NL)],
                           dtype=torch.float64, device="cuda")
    assert (ret_dev.cpu().numpy() == ret).all()
    kept = torch.full((NL, Bsz, H, Cap), -1, dtype=torch.int32, device="cuda")
    dev_err = torch.zeros(1, dtype=torch.int32, device="cuda")
    B.reco_select_compact(cache, torch.from_numpy(sc).cuda(), ret_dev, w, kept_idx=kept, dev_err=dev_err)
    torch.cuda.synchronize()
    assert dev_err.item() == 0
    kk, lc = kept.cpu().numpy(), cache.length.cpu().numpy()
    kc, vc = cache.k.cpu(), cache.v.cpu()
    for u in np.ndindex(NL, Bsz, H):
        l, b, _ = u
        L = int(lens[u])
        ref = oracle.select_unit(sc[u].astype(np.float64), L, w, ret[l, b])
        m = len(ref)
        assert lc[u] == m == oracle.kept_count(L, w, ret[l, b])
        assert (kk[u][:m] == ref).all(), u
        idx = torch.from_numpy(ref)
        assert torch.equal(kc[u][:m], k[u][idx]) and torch.equal(vc[u][:m], v[u][idx])
    assert lc[0, 0, 0] > lc[NL - 1, 0, 0]


@pytest.mark.parametrize("mode,kernel,spread", [("max", 7, 0.0), ("mean", 5, 0.5), ("max", 31, 0.9)])
def test_score_pool_select_pipeline(mode, kernel, spread):
    """Real scores (Eq. 2 on a bf16 cache with heavy hitters) -> pooling ->
    per-layer selection, against the oracle's fp64 pipeline (ties excused)."""
    wl = I.Workload("policy-3L-8q2kv-d128-bf16", n_layers=3, batch=2, n_q_heads=8, n_kv_heads=2, head_dim=128,
                    dtype="bf16", lengths=(3000,), window=32, decode_steps=0, reward="uniform", seed=77)
    ci = I.make_cache(wl, capacity=3000, seq_lens=[3000, 2111])
    cache = B.KVCache(ci.k.cuda(), ci.v.cuda(), ci.length.cuda())
    K, V = f64(ci.k), f64(ci.v)
    lens = ci.length.numpy().astype(np.int64)
    NL, Bsz, H = lens.shape
    scale = 1 / np.sqrt(128)
    base = [0.4, 0.75]
    ret = torch.tensor([[B.reco_layer_retention(r, l, NL, spread) for r in base] for l in range(NL)],
                       dtype=torch.float64, device="cuda")
    dev_err = torch.zeros(1, dtype=torch.int32, device="cuda")
    s = B.reco_score(cache, ci.q_win.cuda(), wl.window, dev_err=dev_err)
    pooled = B.reco_pool_scores(cache, s, wl.window, kernel, mode, dev_err=dev_err)
    kept = torch.full(s.shape, -1, dtype=torch.int32, device="cuda")
    B.reco_select_compact(cache, pooled, ret, wl.window, kept_idx=kept, dev_err=dev_err)
    torch.cuda.synchronize()
    assert dev_err.item() == 0
    s_or = oracle.score_cache(K, lens, f64(ci.q_win), scale)
    kk, lc = kept.cpu().numpy(), cache.length.cpu().numpy()
    kc, vc = cache.k.cpu(), cache.v.cpu()
    for u in np.ndindex(NL, Bsz, H):
        l, b, _ = u
        L = int(lens[u])
        r = oracle.layer_retention(base[b], l, NL, spread)
        p_or = oracle.pool_scores(s_or[u], L, wl.window, kernel, mode)
        ok, msg = kept_sets_match(kk[u], p_or, L, wl.window, r)
        assert ok, (u, msg)
        m = oracle.kept_count(L, wl.window, r)
        assert lc[u] == m
        idx = torch.from_numpy(kk[u][:m].astype(np.int64))
        assert torch.equal(kc[u][:m], ci.k[u][idx]) and torch.equal(vc[u][:m], ci.v[u][idx])
