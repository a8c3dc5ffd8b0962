"""GPU parity of reco_decode_attn against the CPU oracle (decode_cache)."""
import math

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import assert_decode_close, assert_lse_close, f64, upload
from paper_2608_04771_amd import binding as B
from paper_2608_04771_amd import inputs as I

pytestmark = pytest.mark.gpu


def _random_cache(NL, Bsz, H, Cap, D, dtype, lens, seed):
    g = torch.Generator().manual_seed(seed)
    td = torch.float32 if dtype == "f32" else torch.bfloat16
    k = torch.randn((NL, Bsz, H, Cap, D), generator=g).to(td)
    v = torch.randn((NL, Bsz, H, Cap, D), generator=g).to(td)
    ln = torch.tensor(lens, dtype=torch.int32).reshape(NL, Bsz, H)
    return k, v, ln


@pytest.mark.parametrize("dtype,D,G", [("f32", 64, 4), ("f32", 128, 7), ("bf16", 128, 7), ("bf16", 64, 4),
                                       ("bf16", 128, 1), ("bf16", 128, 16), ("f32", 64, 5), ("bf16", 128, 8),
                                       ("f32", 128, 16), ("bf16", 64, 16)])
@pytest.mark.parametrize("append", [False, True])
def test_decode_ragged_units(dtype, D, G, append):
    """Ragged per-unit lengths spanning empty, single-row, tile edges and a
    nearly full unit; every query head compared with the oracle."""
    NL, Bsz, H, Cap = 2, 2, 3, 1100
    lens = [0, 1, 31, 32, 33, 64, 65, 1000, 1099, 517, 250, 7]
    if not append:
        lens[0] = 3                                        # attention over nothing is undefined
    k, v, ln = _random_cache(NL, Bsz, H, Cap, D, dtype, lens, seed=D * 100 + G * 3 + (dtype == "f32"))
    td = k.dtype
    gq = torch.Generator().manual_seed(5)
    q = torch.randn((NL, Bsz, H * G, D), generator=gq).to(td)
    kn = torch.randn((NL, Bsz, H, D), generator=gq).to(td) if append else None
    vn = torch.randn((NL, Bsz, H, D), generator=gq).to(td) if append else None
    cache = B.KVCache(k.cuda(), v.cuda(), ln.cuda())
    dev_err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out, lse = B.reco_decode_attn(cache, q.cuda(), None if kn is None else kn.cuda(),
                                  None if vn is None else vn.cuda(), dev_err=dev_err)
    torch.cuda.synchronize()
    K, V, lens_np = f64(k), f64(v), ln.numpy().astype(np.int64).copy()
    ref_out, ref_lse = oracle.decode_cache(K, V, lens_np, f64(q), 1 / np.sqrt(D),
                                           None if kn is None else f64(kn), None if vn is None else f64(vn))
    assert dev_err.item() == 0
    assert_decode_close(out, ref_out, dtype, f"{dtype} D={D} G={G}")
    assert_lse_close(lse, ref_lse, dtype, f"{dtype} D={D} G={G}")
    if append:
        assert (cache.length.cpu().numpy() == lens_np).all()
        kc, vc = cache.k.cpu(), cache.v.cpu()
        for idx in np.ndindex(NL, Bsz, H):
            n = int(ln[idx])
            assert torch.equal(kc[idx][n], kn[idx]) and torch.equal(vc[idx][n], vn[idx])
            assert torch.equal(kc[idx][:n], k[idx][:n])


def test_decode_append_overflow_is_reported():
    NL, Bsz, H, Cap, D, G = 1, 1, 2, 64, 128, 4
    k, v, ln = _random_cache(NL, Bsz, H, Cap, D, "bf16", [64, 10], seed=3)
    q = torch.randn((NL, Bsz, H * G, D)).to(torch.bfloat16)
    kn = torch.randn((NL, Bsz, H, D)).to(torch.bfloat16)
    vn = torch.randn((NL, Bsz, H, D)).to(torch.bfloat16)
    cache = B.KVCache(k.cuda(), v.cuda(), ln.cuda())
    dev_err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out, _ = B.reco_decode_attn(cache, q.cuda(), kn.cuda(), vn.cuda(), dev_err=dev_err)
    torch.cuda.synchronize()
    assert dev_err.item() == 1
    assert cache.length.cpu().tolist() == [[[64, 11]]]
    # the full unit still attends over its 64 rows plus the new token
    ref, _ = oracle.decode_unit(f64(k)[0, 0, 0], f64(v)[0, 0, 0], 64, f64(q)[0, 0, :G], 1 / np.sqrt(D),
                                f64(kn)[0, 0, 0], f64(vn)[0, 0, 0])
    assert np.abs(f64(out)[0, 0, :G] - ref).max() <= 2e-2


def test_decode_layer_range_touches_only_its_layers():
    NL, Bsz, H, Cap, D, G = 4, 1, 2, 300, 128, 7
    k, v, ln = _random_cache(NL, Bsz, H, Cap, D, "bf16", [200, 150] * 4, seed=4)
    cache = B.KVCache(k.cuda(), v.cuda(), ln.cuda())
    q = torch.randn((2, Bsz, H * G, D)).to(torch.bfloat16)
    kn = torch.randn((2, Bsz, H, D)).to(torch.bfloat16)
    vn = torch.randn((2, Bsz, H, D)).to(torch.bfloat16)
    out, lse = B.reco_decode_attn(cache, q.cuda(), kn.cuda(), vn.cuda(), layer0=1, n_layers=2)
    torch.cuda.synchronize()
    K, V, L = f64(k)[1:3].copy(), f64(v)[1:3].copy(), ln.numpy()[1:3].astype(np.int64).copy()
    ref, rl = oracle.decode_cache(K, V, L, f64(q), 1 / np.sqrt(D), f64(kn), f64(vn))
    assert_decode_close(out, ref, "bf16")
    assert_lse_close(lse, rl, "bf16")
    assert cache.length.cpu().numpy().reshape(-1).tolist() == [200, 150, 201, 151, 201, 151, 200, 150]
    assert torch.equal(cache.k.cpu()[0], k[0]) and torch.equal(cache.k.cpu()[3], k[3])


def test_decode_tiny_workload_64_steps():
    """The tiny fp32 workload: uncompressed cache, 64 decode steps with append."""
    wl = I.WORKLOADS["tiny"]
    ci = I.make_cache(wl)
    qs, ks, vs = I.make_decode_inputs(wl, ci, wl.decode_steps)
    cache = upload(ci)
    K, V = f64(ci.k), f64(ci.v)
    lens = ci.length.numpy().astype(np.int64).copy()
    ws = B.decode_workspace(cache, wl.n_q_heads)
    for s in range(wl.decode_steps):
        out, lse = B.reco_decode_attn(cache, qs[s].cuda(), ks[s].cuda(), vs[s].cuda(), ws=ws)
        ref, rl = oracle.decode_cache(K, V, lens, f64(qs[s]), 1 / np.sqrt(wl.head_dim), f64(ks[s]), f64(vs[s]))
        assert_decode_close(out, ref, "f32", f"step {s}")
        assert_lse_close(lse, rl, "f32", f"step {s}")
    assert (cache.length.cpu().numpy() == lens).all()


@pytest.mark.parametrize("dtype,D,G", [("bf16", 128, 7), ("f32", 64, 4)])
def test_decode_single_unit_max_splits(dtype, D, G):
    """One long unit: the call splits it the maximum 128 ways and merges the
    splits with the many-split merge; appended row and length checked too."""
    NL, Bsz, H, Cap = 1, 1, 1, 20000
    lens = [17001]
    k, v, ln = _random_cache(NL, Bsz, H, Cap, D, dtype, lens, seed=77)
    td = k.dtype
    gq = torch.Generator().manual_seed(6)
    q = torch.randn((NL, Bsz, H * G, D), generator=gq).to(td)
    kn = torch.randn((NL, Bsz, H, D), generator=gq).to(td)
    vn = torch.randn((NL, Bsz, H, D), generator=gq).to(td)
    cache = B.KVCache(k.cuda(), v.cuda(), ln.cuda())
    assert B.decode_attn_workspace_size(cache, H * G) >= 128 * (16 * D + 32) * 4
    dev_err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out, lse = B.reco_decode_attn(cache, q.cuda(), kn.cuda(), vn.cuda(), dev_err=dev_err)
    torch.cuda.synchronize()
    assert dev_err.item() == 0
    n = lens[0]
    ref, rl = oracle.decode_unit(f64(k[0, 0, 0][:n]), f64(v[0, 0, 0][:n]), n, f64(q[0, 0]), 1 / math.sqrt(D),
                                 f64(kn[0, 0, 0]), f64(vn[0, 0, 0]))
    assert_decode_close(out[0, 0], ref, dtype, "single unit")
    assert_lse_close(lse[0, 0], rl, dtype, "single unit")
    assert int(cache.length[0, 0, 0].item()) == n + 1
    assert torch.equal(cache.k[0, 0, 0, n].cpu(), kn[0, 0, 0]) and torch.equal(cache.v[0, 0, 0, n].cpu(), vn[0, 0, 0])


@pytest.mark.parametrize("dtype,D", [("bf16", 128), ("f32", 64)])
def test_decode_empty_unit_without_append(dtype, D):
    """A unit with no rows and no append: output 0, lse -inf, statistics
    (-inf, 0), as the header states; the other units are unaffected."""
    NL, Bsz, H, Cap, G = 1, 1, 2, 64, 4
    k, v, ln = _random_cache(NL, Bsz, H, Cap, D, dtype, [0, 40], seed=3)
    q = torch.randn((NL, Bsz, H * G, D), generator=torch.Generator().manual_seed(4)).to(k.dtype)
    cache = B.KVCache(k.cuda(), v.cuda(), ln.cuda())
    st = torch.empty((NL, Bsz, H * G, 2), dtype=torch.float32, device="cuda")
    dev_err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out, lse = B.reco_decode_attn(cache, q.cuda(), dev_err=dev_err, row_stats=st)
    torch.cuda.synchronize()
    assert dev_err.item() == 0
    assert (out[0, 0, :G].float() == 0).all()
    assert torch.isinf(lse[0, 0, :G]).all() and (lse[0, 0, :G] < 0).all()
    assert torch.isinf(st[0, 0, :G, 0]).all() and (st[0, 0, :G, 1] == 0).all()
    ref, rl = oracle.decode_unit(f64(k[0, 0, 1][:40]), f64(v[0, 0, 1][:40]), 40, f64(q[0, 0, G:]), 1 / math.sqrt(D))
    assert_decode_close(out[0, 0, G:], ref, dtype, "non-empty unit")
    assert_lse_close(lse[0, 0, G:], rl, dtype, "non-empty unit")
    assert cache.length.cpu().tolist() == [[[0, 40]]]


@pytest.mark.parametrize("cap", [64, 512, 4096])
def test_decode_bad_length_is_reported(cap):
    """A stored length below 0 or above capacity sets RECO_DEV_BAD_LENGTH; the
    unit attends over its clamped rows (plus the new token), performs no
    append and keeps its length.  The capacities cover the three completion
    paths: one split finalised in place (64), the one-wave merge of a few
    splits (512) and the many-split merge (4096)."""
    NL, Bsz, H, D, G = 1, 1, 3, 128, 4
    lens = [-3, cap + 5, 20]
    g = torch.Generator().manual_seed(cap)
    k = torch.randn((NL, Bsz, H, cap, D), generator=g).to(torch.bfloat16)
    v = torch.randn((NL, Bsz, H, cap, D), generator=g).to(torch.bfloat16)
    q = torch.randn((NL, Bsz, H * G, D), generator=g).to(torch.bfloat16)
    kn = torch.randn((NL, Bsz, H, D), generator=g).to(torch.bfloat16)
    vn = torch.randn((NL, Bsz, H, D), generator=g).to(torch.bfloat16)
    ln = torch.tensor(lens, dtype=torch.int32).reshape(NL, Bsz, H)
    cache = B.KVCache(k.cuda(), v.cuda(), ln.cuda())
    dev_err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out, _ = B.reco_decode_attn(cache, q.cuda(), kn.cuda(), vn.cuda(), dev_err=dev_err)
    torch.cuda.synchronize()
    assert dev_err.item() == 5
    assert cache.length.cpu().reshape(-1).tolist() == [-3, cap + 5, 21]
    out = out.cpu()
    scale = 1 / math.sqrt(D)
    # length -3: no cached rows, so every head returns the new token's value
    assert torch.equal(out[0, 0, :G], vn[0, 0, 0].expand(G, D))
    # length cap + 5: the cap rows plus the new token
    ref, _ = oracle.decode_unit(f64(k[0, 0, 1]), f64(v[0, 0, 1]), cap, f64(q[0, 0, G:2 * G]), scale,
                                f64(kn[0, 0, 1]), f64(vn[0, 0, 1]))
    assert_decode_close(out[0, 0, G:2 * G], ref, "bf16", f"cap={cap} clamped unit")
    # the valid unit attends and appends as usual
    ref, _ = oracle.decode_unit(f64(k[0, 0, 2]), f64(v[0, 0, 2]), 20, f64(q[0, 0, 2 * G:]), scale,
                                f64(kn[0, 0, 2]), f64(vn[0, 0, 2]))
    assert_decode_close(out[0, 0, 2 * G:], ref, "bf16", f"cap={cap} valid unit")
    kc, vc = cache.k.cpu(), cache.v.cpu()
    assert torch.equal(kc[0, 0, :2], k[0, 0, :2]) and torch.equal(vc[0, 0, :2], v[0, 0, :2])   # no append
    assert torch.equal(kc[0, 0, 2, 20], kn[0, 0, 2]) and torch.equal(vc[0, 0, 2, 20], vn[0, 0, 2])


@pytest.mark.parametrize("units,cap", [(1, 20000), (4, 16640), (112, 16640), (256, 4096), (300, 4096), (4, 100)])
def test_decode_workspace_follows_the_device_compute_units(units, cap):
    """The split count is min(CUs / units, 128, capacity tiles / 4), at least
    1, with the CU count read from the device: the workspace holds one
    partial of 16 x D fp32 + 32 statistics per (unit, split)."""
    D = 128
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    k = torch.zeros((1, 1, units, cap, D), dtype=torch.bfloat16, device="cuda")
    ln = torch.zeros((1, 1, units), dtype=torch.int32, device="cuda")
    cache = B.KVCache(k, k, ln)
    tiles_cap = (cap + 1 + 31) // 32
    splits = max(1, min(cus // units, 128, max(1, tiles_cap // 4)))
    assert B.decode_attn_workspace_size(cache, units * 4) == units * splits * (16 * D + 32) * 4
