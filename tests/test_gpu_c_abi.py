"""The C ABI used from plain C, with no Python binding and no torch on the GPU
side: a C11 program (tests/c_abi/reco_c_driver.c, built by build()) allocates
device memory with the HIP runtime, runs one compression (Eq. 2 scoring, then
selection and in-place compaction, Section 3.2), decode steps that append
their token, the banded reflection penalty (Eq. 3-4) and the answer
perplexity with its stop flag (Eq. 5-6) through libreco.so, and writes its
results to a file.  They are compared here with the oracle under the same
rules as the other GPU tests: scores within SCORE_RTOL (THETA_RTOL near the
k-th value), kept sets equal up to excused ties, decode outputs and
log-sum-exps within the decode tolerances, lengths exact, penalised logits
bit-exact, ln PPL within 1e-5 and the stop flags exact."""
import math
import os
import struct
import subprocess

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import SCORE_RTOL, assert_decode_close, assert_lse_close, assert_theta_precision, kept_sets_match
from paper_2608_04771_amd import inputs as I

pytestmark = pytest.mark.gpu

DRIVER = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "reco_c_driver")

# (workload, sequence lengths or None for the workload's own, decode steps)
TAUS, BETAS, TAU_P = (0.4, 0.8), (0.0, 1.0, 3.0), 1.1

CASES = [
    (I.WORKLOADS["tiny"], None, 8),
    # bf16, head_dim 128, G = 7, ragged sequences over two layers
    (I.Workload("c-abi-2L-14q2kv-d128-bf16", 2, 3, 14, 2, 128, "bf16", (700,), 64, 6, "beta22", 4242,
                vocab=50000),
     (700, 1100, 300), 6),
]


def _raw(t: torch.Tensor) -> bytes:
    t = t.contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().tobytes()
    return t.numpy().tobytes()


def _from_raw(buf: bytes, shape, dtype: str) -> torch.Tensor:
    if dtype == "f32":
        return torch.from_numpy(np.frombuffer(buf, dtype=np.float32).copy().reshape(shape))
    return torch.from_numpy(np.frombuffer(buf, dtype=np.int16).copy().reshape(shape)).view(torch.bfloat16)


@pytest.mark.parametrize("wl,seq_lens,steps", CASES, ids=["tiny-f32", "ragged-bf16"])
def test_c_driver_compress_then_decode(tmp_path, wl, seq_lens, steps):
    if not os.path.exists(DRIVER):
        pytest.fail("tests/c_abi/reco_c_driver is not built: run __graft_entry__.build()")
    ci = I.make_cache(wl, seq_lens=seq_lens)
    NL, Bsz, H, cap, D = ci.k.shape
    Hq, w = wl.n_q_heads, wl.window
    scale = 1.0 / math.sqrt(D)
    r = [oracle.retention_from_reward(float(v)) for v in ci.reward]
    qs, ks, vs = I.make_decode_inputs(wl, ci, steps)
    dt = 0 if wl.dtype == "f32" else 1

    inp = tmp_path / "in.bin"
    with open(inp, "wb") as f:
        f.write(struct.pack("<9i", NL, Bsz, H, Hq, D, cap, w, dt, steps))
        f.write(struct.pack("<f", scale))
        f.write(np.asarray(r, dtype=np.float64).tobytes())
        f.write(ci.length.numpy().astype(np.int32).tobytes())
        for t in (ci.k, ci.v, ci.q_win):
            f.write(_raw(t))
        for seq in (qs, ks, vs):
            for t in seq:
                f.write(_raw(t))
        # Eq. 3-4: one logit row per band edge and its neighbours, 64 reflection ids
        reward = np.array([0.1, 0.4, np.nextafter(np.float32(0.4), np.float32(1)), 0.6,
                           np.nextafter(np.float32(0.8), np.float32(0)), 0.8, 0.95], dtype=np.float32)
        V = wl.vocab
        logits = I.make_logits(len(reward), V, seed=wl.seed + 17).numpy()
        refl = I.make_reflection_ids(wl.n_reflection_ids, V, seed=wl.seed + 19)
        f.write(struct.pack("<3i", len(reward), V, len(refl)))
        f.write(struct.pack("<5f", *TAUS, *BETAS))
        f.write(logits.tobytes())
        f.write(refl.astype(np.int32).tobytes())
        f.write(reward.tobytes())
        # Eq. 5-6: three answers, the second boosted to a confident one (stop branch)
        pb, pn = 3, wl.answer_len
        alog = I.make_logits(pb * pn, V, seed=wl.seed + 23, shape=(pb, pn, V)).numpy()
        atok = I.make_answer_tokens(pb, pn, V, seed=wl.seed + 29)
        alog[1, np.arange(pn), atok[1]] += 25.0
        f.write(struct.pack("<3if", pb, pn, V, TAU_P))
        f.write(alog.tobytes())
        f.write(atok.astype(np.int32).tobytes())
    outp = tmp_path / "out.bin"
    print(f"c driver: {wl.name} NL={NL} B={Bsz} H={H} Hq={Hq} D={D} cap={cap} steps={steps}", flush=True)
    res = subprocess.run([DRIVER, str(inp), str(outp)], capture_output=True, text=True, timeout=90)
    assert res.returncode == 0, f"driver failed ({res.returncode}): {res.stderr[-2000:]}"

    e = 4 if wl.dtype == "f32" else 2
    buf = outp.read_bytes()
    sizes = [4, NL * Bsz * H * cap * 4, NL * Bsz * H * cap * 4, NL * Bsz * H * 4,
             steps * NL * Bsz * Hq * D * e, steps * NL * Bsz * Hq * 4, logits.nbytes, pb * 4, pb * 4]
    assert len(buf) == sum(sizes)
    parts, o = [], 0
    for n in sizes:
        parts.append(buf[o:o + n])
        o += n
    dev_err = struct.unpack("<i", parts[0])[0]
    scores = np.frombuffer(parts[1], dtype=np.float32).reshape(NL, Bsz, H, cap).astype(np.float64)
    kept = np.frombuffer(parts[2], dtype=np.int32).reshape(NL, Bsz, H, cap)
    lens_out = np.frombuffer(parts[3], dtype=np.int32).reshape(NL, Bsz, H)
    outs = _from_raw(parts[4], (steps, NL, Bsz, Hq, D), wl.dtype)
    lses = torch.from_numpy(np.frombuffer(parts[5], dtype=np.float32).copy().reshape(steps, NL, Bsz, Hq))
    pen_out = np.frombuffer(parts[6], dtype=np.float32).reshape(logits.shape)
    ppl = np.frombuffer(parts[7], dtype=np.float32).astype(np.float64)
    stop = np.frombuffer(parts[8], dtype=np.int32)
    assert dev_err == 0

    # Penalty bit-exact; answer perplexity within 1e-5 in ln and the stop flags exact.
    ref_pen = oracle.logit_penalty(logits, refl, reward, *TAUS, *BETAS)
    assert pen_out.tobytes() == ref_pen.tobytes()
    ppl_or, stop_or = oracle.answer_ppl(alog, atok, TAU_P)
    assert np.abs(np.log(ppl) - np.log(ppl_or)).max() <= 1e-5, (ppl, ppl_or)
    assert stop.tolist() == stop_or.astype(int).tolist() and stop_or[1] and not stop_or[0]

    # Compression: scores, then the kept sets (ties excused); the oracle then
    # compacts with the driver's selection so an excused tie cannot diverge.
    K, V = I.to_f64(ci.k), I.to_f64(ci.v)
    lens = ci.length.numpy().astype(np.int64)
    s_or = oracle.score_cache(K, lens, I.to_f64(ci.q_win), scale)
    for u in np.ndindex(NL, Bsz, H):
        L = int(lens[u])
        big = s_or[u][:L] > 1e-20
        rel = np.abs(scores[u][:L] - s_or[u][:L]) / np.maximum(s_or[u][:L], 1e-30)
        assert rel[big].max() <= SCORE_RTOL, (u, float(rel[big].max()))
        assert_theta_precision(scores[u], s_or[u], L, w, r[u[1]], f"c driver unit {u}")
        ok, msg = kept_sets_match(kept[u], s_or[u], L, w, r[u[1]])
        assert ok, (u, msg)
        m = oracle.kept_count(L, w, r[u[1]])
        idx = kept[u][:m]
        K[u][:m], V[u][:m] = oracle.compact_unit(K[u], V[u], idx)
        lens[u] = m
    # Decode steps with append.
    for s in range(steps):
        ref, rl = oracle.decode_cache(K, V, lens, I.to_f64(qs[s]), scale, I.to_f64(ks[s]), I.to_f64(vs[s]))
        assert_decode_close(outs[s], ref, wl.dtype, f"step {s}")
        assert_lse_close(lses[s], rl, wl.dtype, f"step {s}")
    assert (lens_out == lens).all()
