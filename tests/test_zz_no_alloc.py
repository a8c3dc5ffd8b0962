"""The allocation-free decode entry point, reco_decode_attn_noalloc, against
reco_decode_attn through the C ABI: the same inputs on two identical cache
copies, two calls in a row with the second one smaller, and the outputs,
log-sum-exps, row statistics, appended rows and lengths compared.  Both entry
points run the same kernels with the same split count, so everything must
agree bit for bit (stricter than the decode tolerances)."""
import pytest
import torch

from paper_2608_04771_amd import binding as B
from paper_2608_04771_amd import inputs as I

pytestmark = pytest.mark.gpu


def _compare(wl, n_layers, seq_lens, steps, append=True):
    dev = torch.device("cuda")
    print(f"noalloc: {wl.name} layers={n_layers} seq_lens={seq_lens} steps={steps} append={append}", flush=True)
    ci = I.make_cache(wl, device=dev, n_layers=n_layers, seq_lens=seq_lens)
    ref = B.KVCache(ci.k.clone(), ci.v.clone(), ci.length.clone())
    got = B.KVCache(ci.k, ci.v, ci.length)
    qs, ks, vs = I.make_decode_inputs(wl, ci, steps, device=dev)
    NL, Bsz = ci.k.shape[:2]
    Hq = wl.n_q_heads
    err_ref = torch.zeros(1, dtype=torch.int32, device=dev)
    err_got = torch.zeros(1, dtype=torch.int32, device=dev)
    for s in range(steps):
        kn, vn = (ks[s], vs[s]) if append else (None, None)
        rs_ref = torch.empty((NL, Bsz, Hq, 2), dtype=torch.float32, device=dev)
        o_ref, l_ref = B.reco_decode_attn(ref, qs[s], kn, vn, row_stats=rs_ref, dev_err=err_ref)
        o_got = torch.empty_like(qs[s])
        l_got = torch.empty((NL, Bsz, Hq), dtype=torch.float32, device=dev)
        rs_got = torch.empty_like(rs_ref)
        B.reco_decode_attn_noalloc(got, qs[s], o_got, l_got, kn, vn, row_stats=rs_got, dev_err=err_got)
        torch.cuda.synchronize()
        assert torch.equal(o_ref, o_got), f"step {s}: outputs differ"
        assert torch.equal(l_ref, l_got), f"step {s}: lse differs"
        assert torch.equal(rs_ref, rs_got), f"step {s}: row statistics differ"
    assert err_ref.item() == 0 and err_got.item() == 0
    assert torch.equal(ref.length, got.length)
    assert torch.equal(ref.k, got.k) and torch.equal(ref.v, got.v)      # appended rows included
    return int(got.length.max().item())


def test_noalloc_two_calls_second_smaller():
    """7B-shaped bf16 (G = 7, head_dim 128): 8 layers x 5,000 rows (32 units,
    several splits each), then 2 layers x 1,500 rows (8 units) on the same
    static partials array, each with appending decode steps."""
    wl = I.WORKLOADS["7b16k"]
    n1 = _compare(wl, 8, [5000], steps=2)
    n2 = _compare(wl, 2, [1500], steps=2)
    assert n1 == 5002 and n2 == 1502


def test_noalloc_fp32_no_append_and_single_split():
    """fp32 head_dim 64 without append, then a batch whose units are finalised
    in place (one split each: no partials at all)."""
    _compare(I.WORKLOADS["tiny"], 1, [2048], steps=2, append=False)
    wl = I.Workload("noalloc-2L-8q2kv-d128-bf16-B64", 2, 64, 8, 2, 128, "bf16", (300,), 32, 2, "beta22", 4343)
    _compare(wl, 2, [300] * 64, steps=2)


def test_noalloc_many_units_one_split_fallback():
    """More units (512) than compute units, each 8,200 rows long:
    reco_decode_attn cuts every unit in two splits, whose partials (512 x 2 x
    8,320 bytes) would not fit the 8 MiB array, so the allocation-free call
    finalises each unit in one workgroup.  Its outputs then agree with
    reco_decode_attn's and with the oracle's within the bf16 decode
    tolerances; the appended rows and the lengths agree bit for bit."""
    import numpy as np

    import oracle
    from gpu_helpers import assert_decode_close, assert_lse_close, f64

    wl = I.Workload("noalloc-8L-8q1kv-d128-bf16-B64-L8200", 8, 64, 8, 1, 128, "bf16", (8200,), 32, 1, "beta22",
                    4545)
    dev = torch.device("cuda")
    print(f"noalloc fallback: {wl.name}", flush=True)
    ci = I.make_cache(wl, device=dev)
    ref = B.KVCache(ci.k.clone(), ci.v.clone(), ci.length.clone())
    got = B.KVCache(ci.k, ci.v, ci.length)
    qs, ks, vs = I.make_decode_inputs(wl, ci, 1, device=dev)
    NL, Bsz = ci.k.shape[:2]
    err_ref = torch.zeros(1, dtype=torch.int32, device=dev)
    err_got = torch.zeros(1, dtype=torch.int32, device=dev)
    o_ref, l_ref = B.reco_decode_attn(ref, qs[0], ks[0], vs[0], dev_err=err_ref)
    o_got = torch.empty_like(qs[0])
    l_got = torch.empty((NL, Bsz, wl.n_q_heads), dtype=torch.float32, device=dev)
    B.reco_decode_attn_noalloc(got, qs[0], o_got, l_got, ks[0], vs[0], dev_err=err_got)
    torch.cuda.synchronize()
    assert err_ref.item() == 0 and err_got.item() == 0
    assert float((o_ref.float() - o_got.float()).abs().max()) <= 2e-2
    assert float((l_ref - l_got).abs().max()) <= 1e-4
    assert torch.equal(ref.length, got.length) and int(got.length.max().item()) == 8201
    assert torch.equal(ref.k, got.k) and torch.equal(ref.v, got.v)
    scale = 1.0 / np.sqrt(wl.head_dim)
    for (l, b) in [(0, 0), (3, 17), (7, 63)]:
        n = 8201
        o, z = oracle.decode_unit(f64(got.k[l, b, 0, :n]), f64(got.v[l, b, 0, :n]), n, f64(qs[0][l, b]), scale)
        assert_decode_close(o_got[l, b], o, "bf16", f"unit {(l, b)}")
        assert_lse_close(l_got[l, b], z, "bf16", f"unit {(l, b)}")
