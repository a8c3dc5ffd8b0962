"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every entry point the header declares, and rejects invalid arguments before
launching anything.  Validation precedes every HIP call, so these calls are
safe on a machine without a GPU."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2608_04771_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "reco.h")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^[A-Za-z][A-Za-z0-9_ ]*[ *]+(reco_\w+)\(", text, re.M)))


def test_library_exports_every_declared_symbol():
    lib = B.load_library()
    names = _declared()
    assert len(names) >= 13
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(B.EXPORTED)


def test_abi_version_and_status_strings():
    lib = B.load_library()
    assert B.reco_abi_version() == 3
    assert lib.reco_status_str(0) == b"ok"
    assert b"workspace" in lib.reco_status_str(3)
    assert lib.reco_status_str(99) == b"unknown status"


def test_retention_policies_match_oracle():
    for v in np.linspace(0, 1, 41):
        assert B.reco_retention_from_reward(v) == oracle.retention_from_reward(v)
    rng = np.random.default_rng(0)
    for _ in range(100):
        hist = rng.uniform(0, 1, size=rng.integers(1, 20))
        assert B.reco_retention_eq1(hist, 0.25, 0.1) == pytest.approx(oracle.retention_eq1(hist, 0.25, 0.1),
                                                                         rel=0, abs=1e-15)
    assert B.reco_retention_eq1([0.4, 0.4], 0.25, 0.1) == 0.25


@pytest.mark.parametrize("L,w,r", [(2048, 32, 0.75), (16384, 64, 0.5807587504386902), (1001, 32, 0.75),
                                   (7, 32, 0.5), (100, 1, 1.0), (0, 4, 0.5), (1, 1, 0.3)])
def test_kept_count_matches_oracle(L, w, r):
    assert B.reco_kept_count(L, w, r) == oracle.kept_count(L, w, r)


def test_kept_count_rejects_bad_retention():
    assert B.reco_kept_count(100, 8, 0.0) == -1
    assert B.reco_kept_count(100, 8, 1.5) == -1
    assert B.reco_kept_count(100, 8, float("nan")) == -1
    assert B.reco_kept_count(-1, 8, 0.5) == -1


def _fake_cache(**kw):
    d = dict(k=0x1000, v=0x2000, len=0x3000, n_layers=2, batch=1, n_kv_heads=2, capacity=64, head_dim=128,
             dtype=B.RECO_BF16)
    d.update(kw)
    return B.RecoKVCache(d["k"], d["v"], d["len"], d["n_layers"], d["batch"], d["n_kv_heads"], d["capacity"],
                         d["head_dim"], d["dtype"])


P = ctypes.c_void_p


def _score(c, layer0=0, nl=2, q=0x10, hq=4, w=8, scale=0.1, flags=1, stats=0, scores=0x20, ws=0x30, wsb=1 << 30):
    lib = B.load_library()
    return lib.reco_score(ctypes.byref(c), layer0, nl, P(q), hq, w, scale, flags, P(stats) if stats else None,
                          P(scores), P(ws), wsb, None, None)


def test_score_rejects_bad_arguments():
    ok = _fake_cache()
    assert _score(_fake_cache(k=0)) == B.RECO_ERR_INVALID_ARG
    assert _score(ok, q=0) == B.RECO_ERR_INVALID_ARG
    assert _score(ok, scores=0) == B.RECO_ERR_INVALID_ARG
    assert _score(ok, layer0=1, nl=2) == B.RECO_ERR_INVALID_ARG          # past the last layer
    assert _score(ok, nl=0) == B.RECO_ERR_INVALID_ARG
    assert _score(ok, hq=3) == B.RECO_ERR_INVALID_ARG                    # not a multiple of n_kv_heads
    assert _score(ok, w=0) == B.RECO_ERR_INVALID_ARG
    assert _score(ok, w=65) == B.RECO_ERR_INVALID_ARG                    # window beyond capacity
    assert _score(ok, scale=float("nan")) == B.RECO_ERR_INVALID_ARG
    assert _score(ok, flags=2) == B.RECO_ERR_INVALID_ARG
    assert _score(ok, flags=0, stats=0x70) == B.RECO_ERR_INVALID_ARG      # decode statistics are causal
    assert _score(_fake_cache(head_dim=96)) == B.RECO_ERR_UNSUPPORTED
    assert _score(_fake_cache(dtype=7)) == B.RECO_ERR_UNSUPPORTED
    assert _score(ok, ws=0) == B.RECO_ERR_WORKSPACE
    assert _score(ok, wsb=16) == B.RECO_ERR_WORKSPACE
    big = _fake_cache(capacity=100000)
    assert _score(big, hq=2 * 100, w=100) == B.RECO_ERR_UNSUPPORTED      # G*w = 10000 rows > 4096
    assert _score(_fake_cache(capacity=(1 << 29) + 1)) == B.RECO_ERR_UNSUPPORTED   # beyond the score grid


def test_select_compact_rejects_bad_arguments():
    lib = B.load_library()
    c = _fake_cache()

    def call(cache=c, scores=0x20, ret=0x40, stride=0, w=8, idx=None, ws=0x30, wsb=1 << 30, layer0=0, nl=2):
        return lib.reco_select_compact(ctypes.byref(cache), layer0, nl, P(scores), P(ret), stride, w,
                                       P(idx) if idx else None, P(ws), wsb, None, None)
    assert call(scores=0) == B.RECO_ERR_INVALID_ARG
    assert call(ret=0) == B.RECO_ERR_INVALID_ARG
    assert call(stride=-1) == B.RECO_ERR_INVALID_ARG
    assert call(w=0) == B.RECO_ERR_INVALID_ARG
    assert call(w=65) == B.RECO_ERR_INVALID_ARG
    assert call(layer0=-1) == B.RECO_ERR_INVALID_ARG
    assert call(cache=_fake_cache(head_dim=32)) == B.RECO_ERR_UNSUPPORTED
    assert call(ws=0) == B.RECO_ERR_WORKSPACE
    need = lib.reco_select_compact_workspace_size(ctypes.byref(c), 2)
    assert need > 0
    assert call(wsb=need - 1) == B.RECO_ERR_WORKSPACE


def test_pool_scores_rejects_bad_arguments():
    lib = B.load_library()
    c = _fake_cache()
    nbytes = 2 * 1 * 2 * 64 * 4

    def call(cache=c, scores=0x100000, pooled=0x200000, w=8, kernel=5, mode=B.RECO_POOL_MAX, layer0=0, nl=2):
        return lib.reco_pool_scores(ctypes.byref(cache), layer0, nl, w, P(scores), P(pooled), kernel, mode, None, None)
    assert call(scores=0) == B.RECO_ERR_INVALID_ARG
    assert call(pooled=0) == B.RECO_ERR_INVALID_ARG
    assert call(kernel=4) == B.RECO_ERR_INVALID_ARG                      # even
    assert call(kernel=0) == B.RECO_ERR_INVALID_ARG
    assert call(kernel=67) == B.RECO_ERR_INVALID_ARG                     # halo exceeds the LDS stage
    assert call(mode=2) == B.RECO_ERR_INVALID_ARG
    assert call(w=0) == B.RECO_ERR_INVALID_ARG
    assert call(nl=3) == B.RECO_ERR_INVALID_ARG
    assert call(pooled=0x100000 + nbytes - 4) == B.RECO_ERR_INVALID_ARG  # overlapping buffers
    assert call(pooled=0x100000 - nbytes + 4) == B.RECO_ERR_INVALID_ARG


def test_layer_retention_matches_oracle_exactly():
    for NL in (1, 2, 28, 32, 64):
        for r in (0.15, 0.25, 0.5807587504386902, 0.8, 1.0):
            for rho in (0.0, 0.3, 0.5, 0.9):
                for l in range(NL):
                    assert B.reco_layer_retention(r, l, NL, rho) == oracle.layer_retention(r, l, NL, rho)
    import math
    for bad in [(0.0, 0, 4, 0.5), (1.5, 0, 4, 0.5), (0.5, 4, 4, 0.5), (0.5, -1, 4, 0.5), (0.5, 0, 4, 1.0),
                (0.5, 0, 0, 0.5), (0.5, 0, 4, -0.1)]:
        assert math.isnan(B.reco_layer_retention(*bad)), bad


def test_decode_rejects_bad_arguments():
    lib = B.load_library()
    c = _fake_cache()

    def call(cache=c, q=0x10, hq=4, scale=0.1, kn=None, vn=None, out=0x50, ws=0x30, wsb=1 << 30):
        return lib.reco_decode_attn(ctypes.byref(cache), 0, 2, P(q), hq, scale, P(kn) if kn else None,
                                    P(vn) if vn else None, P(out), None, None, P(ws), wsb, None, None)
    assert call(q=0) == B.RECO_ERR_INVALID_ARG
    assert call(out=0) == B.RECO_ERR_INVALID_ARG
    assert call(kn=0x60) == B.RECO_ERR_INVALID_ARG                        # k_new without v_new
    assert call(hq=5) == B.RECO_ERR_INVALID_ARG
    assert call(scale=float("inf")) == B.RECO_ERR_INVALID_ARG
    assert call(hq=2 * 17) == B.RECO_ERR_UNSUPPORTED                      # G = 17 > 16
    assert call(ws=0) == B.RECO_ERR_WORKSPACE
    assert call(wsb=8) == B.RECO_ERR_WORKSPACE


def test_decode_noalloc_rejects_bad_arguments():
    """The allocation-free decode validates exactly like reco_decode_attn
    (every case here is refused before any HIP call)."""
    lib = B.load_library()
    c = _fake_cache()

    def call(cache=c, nl=2, q=0x10, hq=4, scale=0.1, kn=None, vn=None, out=0x50):
        return lib.reco_decode_attn_noalloc(ctypes.byref(cache), 0, nl, P(q), hq, scale, P(kn) if kn else None,
                                            P(vn) if vn else None, P(out), None, None, None, None)
    assert call(q=0) == B.RECO_ERR_INVALID_ARG
    assert call(out=0) == B.RECO_ERR_INVALID_ARG
    assert call(kn=0x60) == B.RECO_ERR_INVALID_ARG                        # k_new without v_new
    assert call(vn=0x60) == B.RECO_ERR_INVALID_ARG
    assert call(nl=3) == B.RECO_ERR_INVALID_ARG
    assert call(hq=5) == B.RECO_ERR_INVALID_ARG
    assert call(scale=float("nan")) == B.RECO_ERR_INVALID_ARG
    assert call(cache=_fake_cache(k=0)) == B.RECO_ERR_INVALID_ARG
    assert call(hq=2 * 17) == B.RECO_ERR_UNSUPPORTED                      # G = 17 > 16
    assert call(cache=_fake_cache(head_dim=96)) == B.RECO_ERR_UNSUPPORTED


def test_penalty_and_ppl_reject_bad_arguments():
    lib = B.load_library()
    pen = lambda logits=0x10, rows=1, vocab=100, ld=100, ids=0x20, n=4, rew=0x30: lib.reco_logit_penalty(  # noqa: E731
        P(logits), rows, vocab, ld, P(ids), n, P(rew), 0.4, 0.8, 0.0, 1.0, 3.0, None, None)
    assert pen(logits=0) == B.RECO_ERR_INVALID_ARG
    assert pen(ld=99) == B.RECO_ERR_INVALID_ARG
    assert pen(n=-1) == B.RECO_ERR_INVALID_ARG
    assert pen(n=5000) == B.RECO_ERR_INVALID_ARG
    assert pen(rew=0) == B.RECO_ERR_INVALID_ARG
    assert pen(n=0, ids=0) == B.RECO_OK                                   # empty set: nothing to do
    assert pen(vocab=(1 << 30) + 1, ld=(1 << 30) + 1) == B.RECO_ERR_UNSUPPORTED
    ppl = lambda logits=0x10, tok=0x20, b=2, n=4, v=100, out=0x30, ws=0x40, wsb=1 << 20: lib.reco_answer_ppl(  # noqa: E731
        P(logits), P(tok), b, n, v, 1.1, P(out), None, P(ws), wsb, None, None)
    assert ppl(logits=0) == B.RECO_ERR_INVALID_ARG
    assert ppl(n=0) == B.RECO_ERR_INVALID_ARG
    assert ppl(out=0) == B.RECO_ERR_INVALID_ARG
    assert ppl(ws=0) == B.RECO_ERR_WORKSPACE
    assert ppl(wsb=4) == B.RECO_ERR_WORKSPACE
    assert ppl(v=(1 << 30) + 1) == B.RECO_ERR_UNSUPPORTED
    assert ppl(b=300, n=300) == B.RECO_ERR_UNSUPPORTED                  # batch * n > 65535


def test_penalty_sample_rejects_bad_arguments():
    lib = B.load_library()
    need = lib.reco_penalty_sample_workspace_size(3, 128256)
    assert need >= 3 * 32 * 8
    assert lib.reco_penalty_sample_workspace_size(0, 10) == 0

    def smp(logits=0x10, rows=3, vocab=128256, ld=128256, ids=0x20, n=4, rew=0x30, T=1.0, tok=0x40, ws=0x50,
            wsb=need):
        return lib.reco_penalty_sample(P(logits), rows, vocab, ld, P(ids), n, P(rew), 0.4, 0.8, 0.0, 1.0, 3.0, T,
                                       2 ** 63 + 5, 2 ** 40, P(tok), P(ws), wsb, None, None)
    assert smp(logits=0) == B.RECO_ERR_INVALID_ARG
    assert smp(tok=0) == B.RECO_ERR_INVALID_ARG
    assert smp(rew=0) == B.RECO_ERR_INVALID_ARG
    assert smp(rows=0) == B.RECO_ERR_INVALID_ARG
    assert smp(rows=65536) == B.RECO_ERR_INVALID_ARG
    assert smp(ld=128255) == B.RECO_ERR_INVALID_ARG
    assert smp(n=4097) == B.RECO_ERR_INVALID_ARG
    assert smp(n=2, ids=0) == B.RECO_ERR_INVALID_ARG
    for bad_t in (-0.5, float("nan"), float("inf"), -0.0 - 1e-30):
        assert smp(T=bad_t) == B.RECO_ERR_INVALID_ARG, bad_t
    assert smp(ws=0) == B.RECO_ERR_WORKSPACE
    assert smp(wsb=need - 1) == B.RECO_ERR_WORKSPACE
    assert smp(vocab=(1 << 30) + 1, ld=(1 << 30) + 1, wsb=1 << 40) == B.RECO_ERR_UNSUPPORTED


def test_workspace_sizes_are_positive_and_monotone():
    lib = B.load_library()
    small, big = _fake_cache(capacity=64), _fake_cache(capacity=4096)
    for fn, args in [("reco_score_workspace_size", (2, 4, 8)), ("reco_decode_attn_workspace_size", (2, 4)),
                     ("reco_select_compact_workspace_size", (2,))]:
        a = getattr(lib, fn)(ctypes.byref(small), *args)
        b = getattr(lib, fn)(ctypes.byref(big), *args)
        assert 0 < a <= b, fn
    assert lib.reco_answer_ppl_workspace_size(8, 32, 152064) >= 8 * 32 * 2 * 4
    assert lib.reco_answer_ppl_workspace_size(0, 32, 10) == 0


def test_workspace_sizes_reject_shapes_the_calls_reject():
    """Sizes are 0 (never an overflowed number) for shapes the entry points
    refuse: too many units for one grid dimension, G * w beyond the score's
    row limit, a score capacity beyond 2^29, a vocabulary beyond 2^30."""
    lib = B.load_library()
    many = _fake_cache(batch=40000, n_kv_heads=2)                        # 80,000 units per layer
    assert lib.reco_score_workspace_size(ctypes.byref(many), 1, 2, 8) == 0
    assert lib.reco_decode_attn_workspace_size(ctypes.byref(many), 1, 2) == 0
    assert lib.reco_select_compact_workspace_size(ctypes.byref(many), 1) == 0
    ok = _fake_cache(capacity=100000)
    assert lib.reco_score_workspace_size(ctypes.byref(ok), 2, 2 * 64, 64) > 0      # G*w = 4096, the limit
    assert lib.reco_score_workspace_size(ctypes.byref(ok), 2, 2 * 65, 64) == 0     # 4160 rows
    assert lib.reco_score_workspace_size(ctypes.byref(ok), 2, 2, 2 ** 31 - 1) == 0
    huge = _fake_cache(capacity=(1 << 29) + 1)                          # beyond the score grid's reach
    assert lib.reco_score_workspace_size(ctypes.byref(huge), 1, 2, 8) == 0
    assert lib.reco_penalty_sample_workspace_size(3, 1 << 30) >= 3 * (1 << 20) * 8
    assert lib.reco_penalty_sample_workspace_size(3, 2 ** 31 - 1) == 0
    assert lib.reco_answer_ppl_workspace_size(1, 1, 2 ** 31 - 1) == 0
