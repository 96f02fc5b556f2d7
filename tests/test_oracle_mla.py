"""Pins of the oracle's decode, combine and BF16 reference.

What fixes each function independently of its own code:
  * decode_none / bf16_reference: torch's scaled-dot-product attention and
    logsumexp on the CPU in float64 (a library routine);
  * decode_streaming vs decode_global: two different statements (the
    Appendix D recurrence and the closed form) must agree;
  * closed forms: one token; zero query with equal scales;
  * a brute-force evaluation with Python loops and the exhaustive encoder;
  * the spec invariants (row sums, scale and permutation invariance)
    and split invariance of the log-sum-exp merge;
  * the P-quantization error bound.
"""

import math

import numpy as np
import pytest
import torch

from oracle import e4m3, mla, quant
from paper_2602_10718_amd import workloads as wl


def _case(seed, R=16, N=200, sigma=1.0, q_len=1, causal=False, H=None):
    rng = np.random.default_rng(seed)
    H = H or R // q_len
    qn = wl.f32_to_bf16_bits(rng.standard_normal((R, 512)).astype(np.float32))
    qr = wl.f32_to_bf16_bits(rng.standard_normal((R, 64)).astype(np.float32))
    ck = rng.standard_normal((N, 512)).astype(np.float32)
    ck *= np.exp(rng.standard_normal(N) * sigma).astype(np.float32)[:, None]
    ck[:, [5, 77, 300, 400]] *= 20
    kr = wl.f32_to_bf16_bits(rng.standard_normal((N, 64)).astype(np.float32))
    ckb = wl.f32_to_bf16_bits(ck)
    q8, sq = quant.quantize_rows(qn)
    c8, sk = quant.quantize_rows(ckb)
    vis = mla.visible_counts(N, q_len, H, causal)
    return dict(q8=q8, sq=sq, qr=qr, c8=c8, sk=sk, kr=kr, qn=qn, ckb=ckb, vis=vis, tau=1 / math.sqrt(192))


def _args(c):
    return (c["q8"], c["sq"], c["qr"], c["c8"], c["sk"], c["kr"], c["tau"], c["vis"])


def _sdpa(c):
    """Library attention on the dequantized cache (float64, CPU)."""
    Q = np.concatenate([e4m3.decode(c["q8"]) * c["sq"].astype(np.float64)[:, None],
                        wl.bf16_bits_to_f32(c["qr"]).astype(np.float64)], axis=1)
    V = e4m3.decode(c["c8"]) * c["sk"].astype(np.float64)[:, None]
    K = np.concatenate([V, wl.bf16_bits_to_f32(c["kr"]).astype(np.float64)], axis=1)
    N = K.shape[0]
    mask = torch.from_numpy(np.arange(N)[None, :] < np.asarray(c["vis"])[:, None])
    q, k, v = (torch.from_numpy(a)[None, None] for a in (Q, K, V))
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=mask[None, None], scale=c["tau"])
    logits = c["tau"] * (torch.from_numpy(Q) @ torch.from_numpy(K).T)
    logits = logits.masked_fill(~mask, -math.inf)
    return o[0, 0].numpy(), torch.logsumexp(logits, dim=1).numpy()


def _rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


@pytest.mark.parametrize("seed,sigma,q_len,causal", [(1, 1.0, 1, False), (2, 1.5, 2, True), (3, 0.3, 1, False)])
def test_decode_none_matches_library_attention(seed, sigma, q_len, causal):
    c = _case(seed, R=16, N=330, sigma=sigma, q_len=q_len, causal=causal)
    o, lse = mla.decode_none(*_args(c))
    o_ref, lse_ref = _sdpa(c)
    assert _rel(o, o_ref) < 1e-12
    assert np.max(np.abs(lse - lse_ref)) < 1e-9 * max(1.0, np.max(np.abs(lse_ref)))


def test_bf16_reference_matches_library_attention():
    c = _case(4, R=8, N=150)
    o, lse = mla.bf16_reference(c["qn"], c["qr"], c["ckb"], c["kr"], c["tau"], c["vis"])
    q = np.concatenate([wl.bf16_bits_to_f32(c["qn"]), wl.bf16_bits_to_f32(c["qr"])], 1).astype(np.float64)
    k = np.concatenate([wl.bf16_bits_to_f32(c["ckb"]), wl.bf16_bits_to_f32(c["kr"])], 1).astype(np.float64)
    v = wl.bf16_bits_to_f32(c["ckb"]).astype(np.float64)
    ot = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None, None], torch.from_numpy(k)[None, None], torch.from_numpy(v)[None, None],
        scale=c["tau"])[0, 0].numpy()
    assert _rel(o, ot) < 1e-12
    lt = torch.logsumexp(c["tau"] * torch.from_numpy(q) @ torch.from_numpy(k).T, dim=1).numpy()
    assert np.max(np.abs(lse - lt)) < 1e-9 * np.max(np.abs(lt))


def test_softmax_rows_sum_to_one():
    c = _case(5, R=32, N=257, q_len=2, causal=True)
    w = mla.softmax_weights(*_args(c))
    assert np.max(np.abs(w.sum(axis=1) - 1)) < 1e-12
    assert np.all(w[:, 256] [:16] == 0)      # the q_len=2 causal mask hides the last token from t=0


@pytest.mark.parametrize("seed,N,q_len,causal", [(6, 1000, 1, False), (7, 333, 2, True), (8, 64, 1, False),
                                                   (9, 65, 2, True)])
def test_streaming_recurrence_equals_closed_form(seed, N, q_len, causal):
    c = _case(seed, R=16, N=N, sigma=1.0, q_len=q_len, causal=causal)
    o1, l1 = mla.decode_streaming(*_args(c))
    o2, l2 = mla.decode_global(*_args(c))
    # blocks far below the row maximum can sit on the EPS floor in one form and
    # not in the other (the floor is relative to a different maximum); their
    # weight is below 1e-10, so the two forms agree to that level
    assert _rel(o1, o2) < 1e-10
    assert np.max(np.abs(l1 - l2)) < 1e-12 * max(1, np.max(np.abs(l2)))


def test_single_token_closed_form():
    c = _case(10, R=8, N=1)
    o, lse = mla.decode_streaming(*_args(c))
    s = mla.logits(c["q8"], c["sq"], c["qr"], c["c8"], c["sk"], c["kr"], c["tau"])[:, 0]
    v = float(c["sk"][0]) * e4m3.decode(c["c8"][0])
    # pi = 448 exactly, so o = sigma_K * D(c8) and LSE = s_0
    assert np.max(np.abs(o - v[None, :])) <= 1e-15 * np.max(np.abs(v))
    assert np.allclose(lse, s, rtol=0, atol=1e-12 * np.max(np.abs(s)))


def test_zero_query_equal_scales_gives_mean():
    c = _case(11, R=4, N=300)
    c["q8"][:] = 0
    c["qr"][:] = 0
    c["sk"][:] = np.float32(0.75)
    o, lse = mla.decode_streaming(*_args(c))
    # all logits 0: every block has et = 0.75 everywhere, pi = 448, o = mean of the values
    mean = 0.75 * e4m3.decode(c["c8"]).mean(axis=0)
    assert np.max(np.abs(o - mean[None, :])) < 1e-13 * np.max(np.abs(mean))
    assert np.allclose(lse, math.log(300), rtol=0, atol=1e-14)


def _brute(c):
    """Python loops + exhaustive encoder: closed form of decode_global for tiny inputs."""
    R, N = c["q8"].shape[0], c["c8"].shape[0]
    tab = e4m3.decode_table()
    o = np.zeros((R, 512))
    lse = np.zeros(R)
    for r in range(R):
        s = []
        for j in range(N):
            acc = 0.0
            for i in range(512):
                acc += tab[c["q8"][r, i]] * tab[c["c8"][j, i]]
            rope = 0.0
            for i in range(64):
                rope += float(wl.bf16_bits_to_f32(c["qr"][r, i:i + 1])[0]) * \
                    float(wl.bf16_bits_to_f32(c["kr"][j, i:i + 1])[0])
            s.append(c["tau"] * (float(c["sq"][r]) * float(c["sk"][j]) * acc + rope))
        M = max(s)
        e = [math.exp(x - M) for x in s]
        lam = sum(e)
        et = [e[j] * float(c["sk"][j]) for j in range(N)]
        for k in range(0, N, 64):
            blk = range(k, min(N, k + 64))
            sP = max(max(et[j] for j in blk) / 448.0, 2.0 ** -40)
            for j in blk:
                pi = int(e4m3.encode_bruteforce(np.array([et[j] / sP]))[0])
                o[r] += sP * tab[pi] * tab[c["c8"][j]]
        o[r] /= lam
        lse[r] = M + math.log(lam)
    return o, lse


def test_bruteforce_tiny():
    for seed, N in ((12, 1), (13, 2), (14, 3), (15, 70)):
        c = _case(seed, R=2, N=N, sigma=1.5)
        ob, lb = _brute(c)
        for fn in (mla.decode_global, mla.decode_streaming):
            o, lse = fn(*_args(c))
            assert _rel(o, ob) < 1e-12
            assert np.max(np.abs(lse - lb)) < 1e-12 * max(1, np.max(np.abs(lb)))


@pytest.mark.parametrize("chunk", [64, 128, 192, 640])
def test_split_invariance(chunk):
    c = _case(16, R=16, N=700, sigma=1.0, q_len=2, causal=True)
    o1, l1 = mla.decode_streaming(*_args(c))
    o2, l2 = mla.decode_split(*_args(c), chunk=chunk)
    # equal up to float64 rounding and EPS-floored blocks of weight < 1e-10
    assert _rel(o2, o1) < 1e-10
    assert np.max(np.abs(l1 - l2)) < 1e-12 * max(1, np.max(np.abs(l1)))


def test_combine_edge_cases():
    o = np.random.default_rng(0).standard_normal((3, 4, 512))
    # lse[part, row]: row 0 has parts 0 and 2, rows 1 and 3 have none, row 2 has all three
    lse = np.array([[0.5, -np.inf, 2.0, -np.inf], [-np.inf, -np.inf, 1.0, -np.inf], [0.1, -np.inf, -3.0, -np.inf]])
    oc, lc = mla.combine(o, lse)
    for r in (1, 3):
        assert np.all(oc[r] == 0) and lc[r] == -np.inf
    assert np.isclose(lc[0], np.logaddexp(0.5, 0.1))
    w = np.exp(lse[[0, 2], 0] - lc[0])
    assert np.allclose(w.sum(), 1) and np.allclose(oc[0], w[0] * o[0, 0] + w[1] * o[2, 0])
    assert np.isclose(lc[2], np.log(np.exp(2.0) + np.exp(1.0) + np.exp(-3.0)))
    o1, l1 = mla.combine(o[:1], lse[:1])
    assert np.array_equal(o1[[0, 2]], o[0, [0, 2]]) and np.array_equal(l1, lse[0])


def test_invisible_row_is_zero_and_minus_inf():
    c = _case(17, R=4, N=100)
    c["vis"] = np.array([0, 100, 1, 64])
    for fn in (mla.decode_streaming, mla.decode_global, mla.decode_none):
        o, lse = fn(*_args(c))
        assert np.all(o[0] == 0) and lse[0] == -np.inf
        assert np.all(np.isfinite(lse[1:]))
    o, lse = mla.decode_streaming(*_args(c))
    v = float(c["sk"][0]) * e4m3.decode(c["c8"][0])
    assert np.max(np.abs(o[2] - v)) <= 1e-15 * np.max(np.abs(v))     # one visible token


def test_scale_invariance_power_of_two():
    # latent value x s and scale x 1/s for s = 2^k: exact without P quantization;
    # with P quantization exact when the token is not its block's largest
    # fused probability and all its codes stay in the normal range.
    c = _case(18, R=8, N=128, sigma=0.5)
    tab = e4m3.decode_table()
    j = 70
    vals = tab[c["c8"][j]]
    # keep the token's codes where x2^k stays exactly representable for |k| <= 2
    ok = ((np.abs(vals) >= 2.0 ** -3) & (np.abs(vals) <= 64)) | (vals == 0)
    c["c8"][j][~ok] = 0
    for k in (1, -1, 2):
        c2 = dict(c)
        c2["c8"] = c["c8"].copy()
        c2["sk"] = c["sk"].copy()
        c2["c8"][j] = e4m3.encode(tab[c["c8"][j]] * 2.0 ** k)
        assert np.array_equal(e4m3.decode(c2["c8"][j]), tab[c["c8"][j]] * 2.0 ** k)
        c2["sk"][j] = np.float32(c["sk"][j] * np.float32(2.0 ** -k))
        o1, l1 = mla.decode_none(*_args(c))
        o2, l2 = mla.decode_none(*_args(c2))
        assert _rel(o2, o1) < 1e-13 and np.max(np.abs(l1 - l2)) < 1e-12
        o1, l1, p1 = mla.decode_global(*_args(c), parts=True)
        o2, l2, p2 = mla.decode_global(*_args(c2), parts=True)
        blk = slice(64, 128)
        notmax = np.all(p1["quot"][:, j] < 448) and np.all(p2["quot"][:, j] < 448)
        normal = np.all(p1["quot"][:, j] * 2.0 ** -k >= 2.0 ** -6) and np.all(p1["quot"][:, j] >= 2.0 ** -6)
        if notmax and normal:
            assert _rel(o2, o1) < 1e-13
        else:
            assert _rel(o2, o1) < 0.07


def test_permutation_invariance():
    c = _case(19, R=8, N=192, sigma=1.0)
    rng = np.random.default_rng(1)
    # within one 64-token block: exact in both modes
    perm = np.arange(192)
    perm[64:128] = 64 + rng.permutation(64)
    c2 = dict(c, c8=c["c8"][perm], sk=c["sk"][perm], kr=c["kr"][perm])
    for fn in (mla.decode_global, mla.decode_none):
        o1, l1 = fn(*_args(c))
        o2, l2 = fn(*_args(c2))
        assert _rel(o2, o1) < 1e-13 and np.max(np.abs(l1 - l2)) < 1e-12
    # across blocks: exact without P quantization, within the P bound with it
    perm = rng.permutation(192)
    c3 = dict(c, c8=c["c8"][perm], sk=c["sk"][perm], kr=c["kr"][perm])
    o1, l1 = mla.decode_none(*_args(c))
    o3, l3 = mla.decode_none(*_args(c3))
    assert _rel(o3, o1) < 1e-13 and np.max(np.abs(l1 - l3)) < 1e-12
    _check_p_bound(c3)


def _check_p_bound(c):
    o8, l8, p = mla.decode_global(*_args(c), parts=True)
    on, ln = mla.decode_none(*_args(c))
    N = c["c8"].shape[0]
    sP = np.repeat(p["sP"], 64, axis=1)[:, :N]
    V = e4m3.decode(c["c8"]) * 1.0
    # each quantized weight sP*D(pi) differs from et by at most 2^-4 et (normal) or 2^-10 sP (subnormal)
    dev = 2.0 ** -4 * p["e"] * c["sk"].astype(np.float64)[None, :] + 2.0 ** -10 * sP
    bound = (dev @ np.abs(V)) / p["lam"][:, None]
    assert np.all(np.abs(o8 - on) <= bound * (1 + 1e-9) + 1e-300)
    assert np.max(np.abs(l8 - ln)) < 1e-12 * max(1, np.max(np.abs(ln)))


@pytest.mark.parametrize("seed,sigma", [(20, 1.0), (21, 1.5), (22, 0.1)])
def test_p_quantization_error_bound(seed, sigma):
    _check_p_bound(_case(seed, R=16, N=500, sigma=sigma))


def test_p_codes_are_block_local():
    # the codes of a block depend only on that block: decode of a prefix chunk
    # reproduces the same codes as the whole sequence (the reference maximum
    # cancels in et / sP).
    c = _case(23, R=8, N=256)
    _, _, p = mla.decode_global(*_args(c), parts=True)
    c2 = dict(c, c8=c["c8"][:128], sk=c["sk"][:128], kr=c["kr"][:128], vis=np.minimum(c["vis"], 128))
    _, _, p2 = mla.decode_global(*_args(c2), parts=True)
    q1, q2 = p["quot"][:, :128], p2["quot"][:, :128]
    fine = p["sP"][:, :2] > 2.0 ** -40
    assert np.allclose(q1[np.repeat(fine, 64, 1)], q2[np.repeat(fine, 64, 1)], rtol=1e-12, atol=0)
