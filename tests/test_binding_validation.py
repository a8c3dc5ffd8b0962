"""The Python binding checks every tensor the C ABI will index before it
calls the library: the ABI receives bare pointers and cannot see extents, so
an undersized or mistyped tensor must be refused here (ValueError), never
passed on.  The caches below live in host memory, so a call whose shapes and
dtypes are all right stops at the device check instead ("must live on the
GPU"): either way nothing reaches the library."""
import pytest
import torch

from paper_2608_04771_amd import binding as B

NL, BS, H, CAP, D, HQ, W = 2, 3, 2, 64, 128, 8, 4
BF, F32, I32, F64 = torch.bfloat16, torch.float32, torch.int32, torch.float64


def _cache(dtype=BF):
    """A KVCache over host tensors (construction skips the device check,
    which every call repeats before touching the library)."""
    c = B.KVCache.__new__(B.KVCache)
    c.k = torch.zeros((NL, BS, H, CAP, D), dtype=dtype)
    c.v = torch.zeros_like(c.k)
    c.length = torch.zeros((NL, BS, H), dtype=I32)
    return c


def _z(*shape, dtype=F32):
    return torch.zeros(shape, dtype=dtype)


def _raises(match, fn, *a, **kw):
    with pytest.raises(ValueError, match=match):
        fn(*a, **kw)


def test_kv_cache_checks_shapes_before_the_device():
    k = _z(NL, BS, H, CAP, D, dtype=BF)
    _raises("k and v", B.KVCache, k, _z(NL, BS, H, CAP, 64, dtype=BF), _z(NL, BS, H, dtype=I32))
    _raises("dtype", B.KVCache, k.half(), k.half(), _z(NL, BS, H, dtype=I32))
    _raises("length", B.KVCache, k, k, _z(NL, BS, H + 1, dtype=I32))
    _raises("length", B.KVCache, k, k, _z(NL, BS, H, dtype=torch.int64))
    _raises("GPU", B.KVCache, k, k, _z(NL, BS, H, dtype=I32))


def test_score_arguments():
    c = _cache()
    q = _z(NL, BS, HQ, W, D, dtype=BF)
    _raises("q_win", B.reco_score, c, _z(NL, BS, HQ, W, D), W)                     # wrong dtype
    _raises("q_win", B.reco_score, c, _z(NL, BS, HQ, W + 1, D, dtype=BF), W)
    _raises("scores", B.reco_score, c, q, W, scores=_z(NL, BS, H, CAP - 1))          # undersized
    _raises("scores", B.reco_score, c, q, W, scores=_z(NL, BS, H, CAP, dtype=F64))
    _raises("row_stats", B.reco_score, c, q, W, row_stats=_z(NL, BS, HQ, W))
    _raises("dev_err", B.reco_score, c, q, W, dev_err=_z(1, dtype=torch.int64))
    _raises("layers", B.reco_score, c, q, W, layer0=1, n_layers=2)
    _raises("GPU", B.reco_score, c, q, W, scores=_z(NL, BS, H, CAP), row_stats=_z(NL, BS, HQ, W, 2))
    # a one-layer call takes one-layer tensors
    _raises("scores", B.reco_score, c, q[1:], W, layer0=1, n_layers=1, scores=_z(NL, BS, H, CAP))
    _raises("GPU", B.reco_score, c, q[1:], W, layer0=1, n_layers=1, scores=_z(1, BS, H, CAP))


def test_select_compact_arguments():
    c = _cache()
    s, r = _z(NL, BS, H, CAP), _z(BS, dtype=F64)
    _raises("retention", B.reco_select_compact, c, s, _z(BS), W)
    _raises("retention", B.reco_select_compact, c, s, _z(BS + 1, dtype=F64), W)
    _raises("scores", B.reco_select_compact, c, _z(NL, BS, H, CAP // 2), r, W)
    _raises("scores", B.reco_select_compact, c, _z(NL, BS, H, CAP, dtype=BF), r, W)
    _raises("kept_idx", B.reco_select_compact, c, s, r, W, kept_idx=_z(NL, BS, H, CAP, dtype=torch.int64))
    _raises("kept_idx", B.reco_select_compact, c, s, r, W, kept_idx=_z(NL, BS, H, 8, dtype=I32))
    _raises("GPU", B.reco_select_compact, c, s, r, W, kept_idx=_z(NL, BS, H, CAP, dtype=I32))
    _raises("GPU", B.reco_select_compact, c, s, _z(NL, BS, dtype=F64), W)          # per-layer budgets


def test_pool_arguments():
    c = _cache()
    s = _z(NL, BS, H, CAP)
    _raises("scores", B.reco_pool_scores, c, _z(NL, BS, H, CAP - 8), W, 5)
    _raises("pooled", B.reco_pool_scores, c, s, W, 5, pooled=_z(NL, BS, H, CAP, dtype=BF))
    _raises("mode", B.reco_pool_scores, c, s, W, 5, mode="median")
    _raises("GPU", B.reco_pool_scores, c, s, W, 5, pooled=_z(NL, BS, H, CAP))


@pytest.mark.parametrize("fn", [B.reco_decode_attn, B.reco_decode_attn_noalloc])
def test_decode_arguments(fn):
    c = _cache()
    q = _z(NL, BS, HQ, D, dtype=BF)
    out = torch.empty_like(q)
    kn = _z(NL, BS, H, D, dtype=BF)

    def call(**kw):
        args = dict(q=q, out=out)
        args.update(kw)
        return fn(c, **args)
    _raises("q must", call, q=_z(NL, BS, HQ, D))                                  # fp32 query into a bf16 cache
    _raises("q must", call, q=_z(NL, BS, HQ, 64, dtype=BF))
    _raises("k_new", call, k_new=kn)                                               # v_new missing
    _raises("k_new", call, k_new=_z(NL, BS, H, D), v_new=kn)                       # fp32 row into a bf16 cache
    _raises("v_new", call, k_new=kn, v_new=_z(NL, BS, H - 1, D, dtype=BF))
    _raises("out", call, out=_z(NL, BS, HQ, D))
    _raises("out", call, out=_z(NL, BS, HQ - 1, D, dtype=BF))
    _raises("lse", call, lse=_z(NL, BS, HQ, 1))
    _raises("row_stats", call, row_stats=_z(NL, BS, HQ, 2, dtype=F64))
    _raises("dev_err", call, dev_err=_z(0, dtype=I32))
    _raises("GPU", call, k_new=kn, v_new=kn, lse=_z(NL, BS, HQ), row_stats=_z(NL, BS, HQ, 2))


def test_decode_noalloc_needs_out():
    c = _cache()
    _raises("out must be given", B.reco_decode_attn_noalloc, c, _z(NL, BS, HQ, D, dtype=BF), None)


def test_logit_arguments():
    z = _z(4, 100)
    ids, rew = _z(8, dtype=I32), _z(4)
    _raises("logits", B.reco_logit_penalty, z.double(), ids, rew, .4, .8, 0., 1., 3.)
    _raises("logits", B.reco_logit_penalty, z.t(), ids, _z(100), .4, .8, 0., 1., 3.)   # column stride != 1
    _raises("refl_ids", B.reco_logit_penalty, z, _z(8, dtype=torch.int64), rew, .4, .8, 0., 1., 3.)
    _raises("reward", B.reco_logit_penalty, z, ids, _z(3), .4, .8, 0., 1., 3.)
    _raises("reward", B.reco_logit_penalty, z, ids, _z(4, dtype=F64), .4, .8, 0., 1., 3.)
    _raises("GPU", B.reco_logit_penalty, z, ids, rew, .4, .8, 0., 1., 3.)
    _raises("tokens", B.reco_penalty_sample, z, ids, rew, .4, .8, 0., 1., 3., 1.0, 0, 0, tokens=_z(3, dtype=I32))
    _raises("tokens", B.reco_penalty_sample, z, ids, rew, .4, .8, 0., 1., 3., 1.0, 0, 0, tokens=_z(4))
    _raises("reward", B.reco_penalty_sample, z, None, _z(5), .4, .8, 0., 1., 3., 1.0, 0, 0)
    _raises("GPU", B.reco_penalty_sample, z, ids, rew, .4, .8, 0., 1., 3., 1.0, 0, 0, tokens=_z(4, dtype=I32))


def test_answer_ppl_arguments():
    z = _z(2, 5, 100)
    tok = _z(2, 5, dtype=I32)
    _raises("logits", B.reco_answer_ppl, _z(10, 100), tok, 1.1)
    _raises("tokens", B.reco_answer_ppl, z, _z(2, 4, dtype=I32), 1.1)
    _raises("tokens", B.reco_answer_ppl, z, _z(2, 5, dtype=torch.int64), 1.1)
    _raises("ppl", B.reco_answer_ppl, z, tok, 1.1, ppl=_z(1))
    _raises("stop", B.reco_answer_ppl, z, tok, 1.1, stop=_z(2))
    _raises("GPU", B.reco_answer_ppl, z, tok, 1.1, ppl=_z(2), stop=_z(2, dtype=I32))


def test_prepared_decode_checks_its_fixed_buffers():
    c = _cache()
    out = _z(NL, BS, HQ, D, dtype=BF)
    lse = _z(NL, BS, HQ)
    ws = _z(1 << 20, dtype=torch.uint8)
    _raises("out", B.PreparedDecode, c, HQ, _z(NL, BS, HQ, D), lse, ws)                 # wrong dtype
    _raises("out", B.PreparedDecode, c, HQ, _z(NL, BS, HQ - 1, D, dtype=BF), lse, ws)
    _raises("lse", B.PreparedDecode, c, HQ, out, _z(NL, BS, HQ + 1), ws)
    _raises("dev_err", B.PreparedDecode, c, HQ, out, lse, ws, dev_err=_z(1, dtype=torch.int64))
    _raises("must be given", B.PreparedDecode, c, HQ, out, lse, None)
    _raises("layers", B.PreparedDecode, c, HQ, out, lse, ws, layer0=2)
    _raises("GPU", B.PreparedDecode, c, HQ, out, lse, ws)


def test_prepared_penalty_sample_checks_its_fixed_buffers():
    rows, vocab = 4, 1000
    ids = _z(8, dtype=I32)
    rew = _z(rows)
    tok = _z(rows, dtype=I32)
    ws = _z(1 << 16, dtype=torch.uint8)
    _raises("refl_ids", B.PreparedPenaltySample, rows, vocab, _z(8), rew, tok, ws)
    _raises("reward", B.PreparedPenaltySample, rows, vocab, ids, _z(rows + 1), tok, ws)
    _raises("tokens", B.PreparedPenaltySample, rows, vocab, ids, rew, _z(rows, dtype=torch.int64), ws)
    _raises("must be given", B.PreparedPenaltySample, rows, vocab, ids, rew, tok, None)
    _raises("GPU", B.PreparedPenaltySample, rows, vocab, ids, rew, tok, ws)
