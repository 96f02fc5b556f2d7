"""Pins of the granularity ablation's oracle (oracle/granularity.py) and the mechanisms it shows."""

import numpy as np
import pytest

from oracle import e4m3, granularity as gr, mla, quant
from paper_2602_10718_amd.workloads import f32_to_bf16_bits, bf16_bits_to_f32
from paper_2602_10718_amd import workloads as wl


def _seq(rng, n, scale=1.0, rope=1.0):
    c = (rng.standard_normal((n, 512)) * scale).astype(np.float32)
    r = (rng.standard_normal((n, 64)) * rope).astype(np.float32)
    return f32_to_bf16_bits(c), f32_to_bf16_bits(r)


def _recon(codes, sigma):
    return e4m3.decode(codes) * sigma.astype(np.float64)[:, None]


def test_snapmla_is_the_per_token_quantizer():
    rng = np.random.default_rng(1)
    seqs = [_seq(rng, 100), _seq(rng, 37, 5.0)]
    for (c, r), (codes, sig, rb) in zip(seqs, gr.quantize("snapmla", seqs)):
        c2, s2 = quant.quantize_rows(c)
        assert np.array_equal(codes, c2) and np.array_equal(sig, s2) and np.array_equal(rb, r)


def test_scales_by_closed_form():
    rng = np.random.default_rng(2)
    seqs = [_seq(rng, 130, 2.0, 50.0), _seq(rng, 64, 0.5, 50.0)]
    x = [bf16_bits_to_f32(c) for c, _ in seqs]
    # C: one scale, the batch amax / 448
    allmax = max(float(np.max(np.abs(v))) for v in x)
    for _, sig, _ in gr.quantize("C", seqs):
        assert np.all(sig == np.float32(np.float32(allmax) / np.float32(448)))
    # D: one scale per 64-token page, that page's amax / 448 (the partial last page included)
    (_, sig, _), _ = gr.quantize("D", seqs)
    for k0 in (0, 64, 128):
        blk = x[0][k0:k0 + 64]
        assert np.all(sig[k0:k0 + 64] == np.float32(np.float32(np.max(np.abs(blk))) / np.float32(448)))
    # A: per token over content and RoPE together; RoPE dominates here
    (codes, sig, rb), _ = gr.quantize("A", seqs)
    r = bf16_bits_to_f32(seqs[0][1])
    amax = np.maximum(np.max(np.abs(x[0]), axis=1), np.max(np.abs(r), axis=1))
    assert np.array_equal(sig, (amax / np.float32(448)).astype(np.float32))
    # the token amax (a RoPE element) reconstructs to itself up to one bf16 rounding
    rq = bf16_bits_to_f32(rb).astype(np.float64)
    j = np.argmax(np.abs(r), axis=1)
    top = rq[np.arange(len(j)), j]
    assert np.all(np.abs(top - r[np.arange(len(j)), j]) <= 2.0 ** -8 * np.abs(r[np.arange(len(j)), j]))
    # and every RoPE element within E4M3's half ulp (2^-4 relative, 2^-10 sigma below the normal range) + bf16
    err = np.abs(rq - r)
    assert np.all(err <= (2.0 ** -4 + 2.0 ** -7) * np.abs(r) + 2.0 ** -10 * sig[:, None] * 1.01)


def test_static_scale_saturates_at_448():
    rng = np.random.default_rng(3)
    c, r = _seq(rng, 10, 300.0)
    (codes, sig, _), = gr.quantize("B", [(c, r)])
    assert np.all(sig == 1.0)
    x = bf16_bits_to_f32(c)
    big = np.abs(x) >= 464
    assert big.any() and np.all((codes[big] & 0x7F) == 0x7E)          # saturated to +-448
    small = np.abs(x) < 448
    assert np.all(np.abs(_recon(codes, sig)[small] - x[small]) <= 2.0 ** -4 * np.abs(x[small]) + 2.0 ** -10)


def test_scores_by_hand():
    ref = np.array([[1.0, 0.0], [0.0, 2.0]])
    o = np.array([[1.0, 1.0], [0.0, 2.0]])
    s = gr.scores(o, ref)
    assert s["rmse"] == pytest.approx(0.5)
    assert s["cos_diff"] == pytest.approx((1 - 1 / np.sqrt(2)) / 2)
    assert s["rel_l2"] == pytest.approx(1 / np.sqrt(5))
    assert gr.scores(ref, ref) == {"rmse": 0.0, "cos_diff": 0.0, "rel_l2": 0.0}


def _attention_error(config, seqs, qn, qr, tau=1 / np.sqrt(192), pquant=True):
    """rel-L2 of the decode over the config's cache against BF16 attention; pquant=False leaves the
    probabilities unquantized (mla.decode_none) to isolate the cache quantization."""
    outs, refs = [], []
    f = mla.decode_global if pquant else mla.decode_none
    for (c, r), (codes, sig, rb), q_n, q_r in zip(seqs, gr.quantize(config, seqs), qn, qr):
        vis = mla.visible_counts(c.shape[0], 1, q_n.shape[0], False)
        q8, sq = quant.quantize_rows(q_n)
        outs.append(f(q8, sq, q_r, codes, sig, rb, tau, vis)[0])
        refs.append(mla.bf16_reference(q_n, q_r, c, r, tau, vis)[0])
    return gr.scores(np.concatenate(outs), np.concatenate(refs))["rel_l2"]


def _queries(rng, B, H, qn_scale=0.1, qr_scale=1.0):
    qn = [f32_to_bf16_bits((rng.standard_normal((H, 512)) * qn_scale).astype(np.float32)) for _ in range(B)]
    qr = [f32_to_bf16_bits((rng.standard_normal((H, 64)) * qr_scale).astype(np.float32)) for _ in range(B)]
    return qn, qr


def test_mechanism_shared_scale_flushes_quiet_tokens():
    """Quiet tokens (magnitude 2^-16) interleaved with loud ones in every block, and queries that
    attend to the quiet ones (through the RoPE term): one scale per tensor (C) or per block (D)
    pushes the quiet tokens below E4M3's range and the output is lost, while per-token scales keep
    every token at full relative precision."""
    rng = np.random.default_rng(4)
    seqs, qn, qr = [], [], []
    for _ in range(2):
        n = 256
        quiet = (np.arange(n) % 2) == 1
        c = rng.standard_normal((n, 512)).astype(np.float32)
        c[quiet] *= np.float32(2.0 ** -16)
        rk = rng.standard_normal((n, 64)).astype(np.float32)
        rk[quiet] += np.float32(3.0)                      # the quiet tokens share a RoPE direction
        seqs.append((f32_to_bf16_bits(c), f32_to_bf16_bits(rk)))
        qn.append(f32_to_bf16_bits((rng.standard_normal((8, 512)) * 0.1).astype(np.float32)))
        qr.append(f32_to_bf16_bits(np.full((8, 64), 1.0, np.float32)))   # ... which the queries favour
    e = {k: _attention_error(k, seqs, qn, qr, pquant=False) for k in ("snapmla", "C", "D")}
    assert e["snapmla"] < 0.1 and e["C"] > 8 * e["snapmla"] and e["D"] > 8 * e["snapmla"], e


def test_mechanism_rope_unaware_loses_the_content():
    """RoPE values 10^6 above the content: a scale shared by both parts (A) pushes the whole
    content below E4M3's range, while RoPE-aware per-token scaling keeps it."""
    rng = np.random.default_rng(5)
    seqs = [_seq(rng, 256, 1.0, 1e6) for _ in range(2)]
    qn, qr = _queries(rng, 2, 8, qn_scale=0.3, qr_scale=1e-7)
    e = {k: _attention_error(k, seqs, qn, qr, pquant=False) for k in ("snapmla", "A")}
    assert e["snapmla"] < 0.1 and e["A"] > 0.5, e


def test_paper_like_regime_static_scale_collapses():
    """The ablation workload (content ~10^0-10^1 with x20 outliers, RoPE ~10^3): the static scale
    saturates the outlier channels; the other granularities stay within a factor 2.5 of per-token."""
    w = wl.ablation(B=2, H=8, ctx=1024)
    qn, qr = w.queries()
    seqs = [w.tokens(b, 0, int(w.seq_lens[b])) for b in range(w.B)]
    qn = [qn[b].reshape(-1, 512) for b in range(w.B)]
    qr = [qr[b].reshape(-1, 64) for b in range(w.B)]
    e = {k: _attention_error(k, seqs, qn, qr) for k in gr.CONFIGS}
    print({k: f"{v:.3e}" for k, v in e.items()})
    assert e["B"] > 5 * e["snapmla"]
    assert all(e[k] < 2.5 * e["snapmla"] for k in ("A", "C", "D")), e
