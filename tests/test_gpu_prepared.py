"""The binding's prepared per-token calls (PreparedDecode,
PreparedPenaltySample) against the plain entry points: the same inputs give
bit-identical outputs, appended rows, lengths, statistics, penalised logits
and tokens, and a tensor of the wrong shape, dtype or device is refused
before anything is launched (the cache is left as it was)."""
import pytest
import torch

from paper_2608_04771_amd import binding as B
from paper_2608_04771_amd import inputs as I

pytestmark = pytest.mark.gpu


def test_prepared_decode_matches_reco_decode_attn():
    wl = I.WORKLOADS["7b16k"]
    dev = torch.device("cuda")
    ci = I.make_cache(wl, device=dev, n_layers=3, seq_lens=[1000])
    ref = B.KVCache(ci.k.clone(), ci.v.clone(), ci.length.clone())
    got = B.KVCache(ci.k, ci.v, ci.length)
    qs, ks, vs = I.make_decode_inputs(wl, ci, 4, device=dev)
    NL, Bsz = ci.k.shape[:2]
    Hq = wl.n_q_heads
    out = torch.empty_like(qs[0])
    lse = torch.empty((NL, Bsz, Hq), dtype=torch.float32, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    call = B.PreparedDecode(got, Hq, out, lse, B.decode_workspace(got, Hq), err)
    for s in range(4):
        st_ref = torch.empty((NL, Bsz, Hq, 2), dtype=torch.float32, device=dev)
        st_got = torch.empty_like(st_ref)
        o_ref, l_ref = B.reco_decode_attn(ref, qs[s], ks[s], vs[s], row_stats=st_ref)
        call(qs[s], ks[s], vs[s], st_got)
        torch.cuda.synchronize()
        assert torch.equal(o_ref, out) and torch.equal(l_ref, lse) and torch.equal(st_ref, st_got)
    assert err.item() == 0
    assert torch.equal(ref.length, got.length) and torch.equal(ref.k, got.k) and torch.equal(ref.v, got.v)
    before = got.length.clone()
    with pytest.raises(ValueError, match="q must be"):
        call(qs[0][:2], ks[0], vs[0])
    with pytest.raises(ValueError, match="q must be"):
        call(qs[0].float(), ks[0], vs[0])
    with pytest.raises(ValueError, match="k_new must be"):
        call(qs[0], ks[0][:, :, :1], vs[0])
    with pytest.raises(ValueError, match="together"):
        call(qs[0], ks[0], None)
    with pytest.raises(ValueError, match="row_stats must be"):
        call(qs[0], ks[0], vs[0], torch.empty((NL, Bsz, Hq), dtype=torch.float32, device=dev))
    with pytest.raises(ValueError, match="q must be"):
        call(qs[0].cpu(), ks[0], vs[0])
    torch.cuda.synchronize()
    assert torch.equal(got.length, before)


def test_prepared_penalty_sample_matches_reco_penalty_sample():
    dev = torch.device("cuda")
    rows, vocab = 3, 50000
    ids = torch.from_numpy(I.make_reflection_ids(64, vocab, seed=5)).to(dev)
    reward = torch.tensor([0.1, 0.5, 0.9], dtype=torch.float32, device=dev)
    tokens = torch.empty(rows, dtype=torch.int32, device=dev)
    ws = torch.empty(B.penalty_sample_workspace_size(rows, vocab), dtype=torch.uint8, device=dev)
    call = B.PreparedPenaltySample(rows, vocab, ids, reward, tokens, ws)
    for offset in (0, 7, 12345):
        z = I.make_logits(rows, vocab, seed=offset + 1, device=dev)
        z_ref = z.clone()
        t_ref = B.reco_penalty_sample(z_ref, ids, reward, 0.4, 0.8, 0.0, 1.0, 3.0, 1.0, 99, offset)
        call(z, 0.4, 0.8, 0.0, 1.0, 3.0, 1.0, 99, offset)
        torch.cuda.synchronize()
        assert torch.equal(t_ref, tokens) and torch.equal(z_ref, z)
    with pytest.raises(ValueError, match="logits must be"):
        call(torch.zeros((rows, vocab - 1), device=dev), 0.4, 0.8, 0.0, 1.0, 3.0, 1.0, 99, 0)
    with pytest.raises(ValueError, match="logits must be"):
        call(torch.zeros((rows, vocab), device=dev, dtype=torch.float64), 0.4, 0.8, 0.0, 1.0, 3.0, 1.0, 99, 0)


def test_prepared_decode_in_a_graph_replays_match_eager():
    """Per-layer prepared calls (no append) captured in a HIP graph: every
    replay, with eager work between replays, equals the eager calls bit for
    bit."""
    wl = I.WORKLOADS["7b16k"]
    dev = torch.device("cuda")
    ci = I.make_cache(wl, device=dev, n_layers=4, seq_lens=[2500])
    cache = B.KVCache(ci.k, ci.v, ci.length)
    NL, Bsz, H, Cap, D = cache.shape
    Hq = wl.n_q_heads
    g = torch.Generator(device="cuda").manual_seed(11)
    q = torch.randn((NL, Bsz, Hq, D), device=dev, generator=g).to(torch.bfloat16)
    ws = torch.empty(B.decode_attn_workspace_size(cache, Hq, 1), dtype=torch.uint8, device=dev)
    out = torch.empty_like(q)
    lse = torch.empty((NL, Bsz, Hq), dtype=torch.float32, device=dev)
    calls = [B.PreparedDecode(cache, Hq, out[l:l + 1], lse[l:l + 1], ws, layer0=l, n_layers=1) for l in range(NL)]

    def per_layer():
        for l in range(NL):
            calls[l](q[l:l + 1])

    per_layer()
    torch.cuda.synchronize()
    ref_out, ref_lse = out.clone(), lse.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        per_layer()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        per_layer()
    for rep in range(3):
        out.zero_()
        lse.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref_out), f"replay {rep}: out differs"
        assert torch.equal(lse, ref_lse), f"replay {rep}: lse differs"
        B.reco_decode_attn(cache, q)                                # eager work between replays
        torch.cuda.synchronize()
    assert (cache.length.cpu().numpy() == 2500).all()
