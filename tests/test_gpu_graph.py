"""Decode calls captured in a HIP graph (the per-layer form a model uses):
every replay, with eager work and synchronisations between replays, must
equal the eager result bit for bit (the launch configuration and the merge
order are the same, and no call records a memset)."""
import numpy as np
import pytest
import torch

from paper_2608_04771_amd import binding as B
from paper_2608_04771_amd import inputs as I

pytestmark = pytest.mark.gpu


def test_per_layer_decode_graph_replays_match_eager():
    wl = I.WORKLOADS["7b16k"]
    ci = I.make_cache(wl, device=torch.device("cuda"), n_layers=4, seq_lens=[3000])
    cache = B.KVCache(ci.k, ci.v, ci.length)
    NL, Bsz, H, Cap, D = cache.shape
    g = torch.Generator(device="cuda").manual_seed(3)
    q = torch.randn((NL, Bsz, wl.n_q_heads, D), device="cuda", generator=g).to(torch.bfloat16)
    ws = torch.empty(B.decode_attn_workspace_size(cache, wl.n_q_heads, 1), dtype=torch.uint8, device="cuda")
    out = torch.empty_like(q)
    lse = torch.empty(q.shape[:3], dtype=torch.float32, device="cuda")

    def per_layer():
        for l in range(NL):
            B.reco_decode_attn(cache, q[l:l + 1], out=out[l:l + 1], lse=lse[l:l + 1], layer0=l, n_layers=1, ws=ws)

    per_layer()
    torch.cuda.synchronize()
    ref_out, ref_lse = out.clone(), lse.clone()
    all_out, all_lse = B.reco_decode_attn(cache, q)                 # one call over all layers
    torch.cuda.synchronize()
    assert (all_out.float() - ref_out.float()).abs().max().item() <= 2e-2
    assert (all_lse - ref_lse).abs().max().item() <= 1e-4

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
    assert (cache.length.cpu().numpy() == 3000).all()
