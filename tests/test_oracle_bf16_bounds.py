"""Pins of the BF16-path bound (oracle/check.bounds_bf16): it holds for a float32 emulation of the
BF16 decode (P rounded to bf16 per 32-token block, online rescaling) and fails for planted mistakes."""

import numpy as np
import pytest

from oracle import check, fetch, quant
from paper_2602_10718_amd import workloads as wl


def _emulate(ref, block=32, round_p=True, drop_rope=False):
    """float32 online-softmax decode over bf16 inputs, P rounded to bf16 before the PV product."""
    Q = quant.bf16_to_f32(ref["qn"])
    Qr = quant.bf16_to_f32(ref["qr"])
    C = quant.bf16_to_f32(ref["ckv"])
    Kr = quant.bf16_to_f32(ref["kr"])
    R, N = Q.shape[0], C.shape[0]
    tau = np.float32(ref["tau"])
    m = np.full(R, -np.inf, np.float32)
    l = np.zeros(R, np.float32)
    O = np.zeros((R, 512), np.float32)
    for j0 in range(0, N, block):
        j1 = min(N, j0 + block)
        s = (Q @ C[j0:j1].T).astype(np.float32)
        if not drop_rope:
            s = (s + Qr @ Kr[j0:j1].T).astype(np.float32)
        s = (s * tau).astype(np.float32)
        s = np.where(np.arange(j0, j1)[None, :] < np.asarray(ref["vis"])[:, None], s, -np.inf).astype(np.float32)
        mb = np.max(s, axis=1)
        m_new = np.maximum(m, mb)
        ok = m_new > -np.inf
        with np.errstate(invalid="ignore"):
            p = np.where(ok[:, None], np.exp(s - np.where(ok, m_new, 0)[:, None]), 0).astype(np.float32)
            g = np.where(ok, np.exp(np.where(ok, m - m_new, 0)), 1).astype(np.float32)
        l = (g * l + p.sum(axis=1)).astype(np.float32)
        pr = (fetch.f32_to_bf16_bits(p).astype(np.uint32) << 16).view(np.float32) if round_p else p
        O = (g[:, None] * O + pr @ C[j0:j1]).astype(np.float32)
        m = np.where(ok, m_new, m)
    o = np.where(l[:, None] > 0, O / np.where(l > 0, l, 1)[:, None], 0)
    return o


@pytest.mark.parametrize("seed", [0, 1])
def test_bound_holds_for_float32_emulation(seed):
    # peaked attention (a few dominant tokens)
    w = wl.custom(B=1, H=16, q_len=1, seq_lens=[700], rotary=True, sigma_tok=1.5, seed=50 + seed)
    ck, kr = w.tokens(0, 0, 700)
    qn, qr = w.queries()
    ref = check.sequence_reference_bf16(qn[0], qr[0], ck, kr, w.tau, 1, 16, False)
    ob, _ = check.bounds_bf16(ref)
    assert np.all(np.abs(_emulate(ref) - ref["o"]) <= ob)


@pytest.mark.parametrize("seed", [0, 1])
def test_bound_is_tight_on_spread_attention(seed):
    # logits spread over a few units: the bf16 rounding of P is the dominant error and uses a
    # sizeable part of the bound, so the bound is not vacuous
    w = wl.ablation(B=1, H=16, ctx=700, seed=1300 + seed)
    ck, kr = w.tokens(0, 0, 700)
    qn, qr = w.queries()
    ref = check.sequence_reference_bf16(qn[0], qr[0], ck, kr, w.tau, 1, 16, False)
    ob, _ = check.bounds_bf16(ref)
    o = _emulate(ref)
    ratio = np.max(np.abs(o - ref["o"]) / ob)
    assert ratio <= 1.0
    assert ratio > 0.05
    # without the P rounding the error is far smaller
    assert np.max(np.abs(_emulate(ref, round_p=False) - ref["o"])) < 0.1 * np.max(np.abs(o - ref["o"]))


def test_bound_catches_planted_mistake():
    w = wl.ablation(B=1, H=16, ctx=700, seed=1310)
    ck, kr = w.tokens(0, 0, 700)
    qn, qr = w.queries()
    ref = check.sequence_reference_bf16(qn[0], qr[0], ck, kr, w.tau, 1, 16, False)
    ob, _ = check.bounds_bf16(ref)
    bad = _emulate(ref, drop_rope=True)              # forgetting the RoPE term of the logits
    assert np.any(np.abs(bad - ref["o"]) > ob)
