"""Host checks of bench.py's accounting: the algorithmic bytes of a
compression and of a decode call, the moved-row count, the roofline object,
and the oracle-rate helpers on small inputs (no GPU)."""
import math

import numpy as np
import pytest
import torch

import bench


def test_decode_call_bytes_counts_rows_queries_and_append():
    # 3 units of 10 attended rows each, 6 query rows, D = 4, bf16
    D, e = 4, 2
    got = bench.decode_call_bytes(30, 3, 6, D, e)
    assert got == 30 * 2 * D * e + 2 * 6 * D * e + 6 * 4 + 2 * 3 * D * e


def test_compress_bytes_one_pass_and_two_pass():
    lens0 = np.full((2, 1, 2), 100, dtype=np.int64)
    m = np.full((2, 1, 2), 60, dtype=np.int64)
    Bsz, Hq, w, D, e = 1, 4, 8, 16, 2
    two = bench.compress_bytes(lens0, m, 50, Bsz, Hq, w, D, e)
    one = bench.compress_bytes(lens0, m, 50, Bsz, Hq, w, D, e, stats_fed=True)
    rows = 400
    assert two["score"] == rows * D * e + 2 * Bsz * Hq * w * D * e + rows * 4
    assert one["score"] - two["score"] == 2 * Bsz * Hq * w * 8      # the (max, sum) of every window row
    assert two["select"] == rows * 4 + 240 * 4
    assert two["compact"] == 50 * 2 * 2 * D * e


def test_moved_rows_counts_positions_that_change():
    kept = torch.zeros((1, 1, 2, 8), dtype=torch.int32)
    kept[0, 0, 0, :5] = torch.tensor([0, 1, 2, 3, 4])        # nothing moves
    kept[0, 0, 1, :5] = torch.tensor([0, 2, 3, 6, 7])        # four rows move
    m = np.array([[[5, 5]]])
    assert bench.moved_rows_of(kept, m) == 4


def test_roofline_object():
    r = bench.roofline_obj("k", 8e9, 2.0)
    assert r["achieved"] == pytest.approx(4000.0)
    assert r["frac"] == pytest.approx(0.5)
    assert r["peak"] == bench.PEAK_HBM_GBPS and r["unit"] == "GB/s" and r["bound"] == "hbm"


def test_oracle_unit_rates_on_small_units():
    rng = np.random.default_rng(0)
    K, V = rng.standard_normal((300, 16)), rng.standard_normal((300, 16))
    Q = rng.standard_normal((2, 8, 16))

    def comp():
        while True:
            yield K, V, Q, 0.5

    def dec():
        while True:
            yield K[:200], V[:200], 200, Q[:, 0], K[0], V[0]
    rt = bench.oracle_unit_rates(comp(), dec(), 1 / math.sqrt(16), 8, 0.05, 0.05)
    assert rt["units_compressed"] >= 1 and rt["decode_samples"] >= 1
    assert rt["s_per_row_compress"] > 0 and rt["s_per_row_decode"] > 0


def test_host_threads_within_affinity():
    threads, affinity = bench.host_threads()
    assert 1 <= threads <= affinity


def test_cpu_baseline_trajectory_runs_the_oracle_on_the_start():
    import dataclasses
    from paper_2608_04771_amd import inputs as I
    wl = dataclasses.replace(I.WORKLOADS["8b-trajectory"], n_layers=1, decode_steps=40)
    ci = I.make_cache(wl, capacity=600)
    prompt = int(ci.seq_len[0])
    k0, v0 = ci.k[..., :prompt, :].clone(), ci.v[..., :prompt, :].clone()
    qs, ks, vs = I.make_decode_inputs(wl, ci, 40)
    qa, ka, va = torch.stack(qs), torch.stack(ks), torch.stack(vs)
    bounds = {10, 25, 40}
    rewards = I.make_rewards("beta25", 3, 1, 5)
    res = bench.cpu_baseline_trajectory(wl, ci, k0, v0, prompt, qa, ka, va, bounds, rewards, wl.window,
                                        budget_s=0.5)
    assert res["kind"] == "oracle" and res["value"] > 0 and res["cores"] >= 1
    assert "generated tokens" in res["sample"]
