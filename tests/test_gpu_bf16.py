"""GPU: the BF16-cache decode (snapmla_decode_bf16 + snapmla_combine) and its append against the
oracle's float64 attention on the bf16 inputs, within the derived BF16-path bounds."""

import numpy as np
import pytest
import torch

from paper_2602_10718_amd import workloads as wl
from gpu_common import runner, reference, reference_bf16, check_sequence_bf16

pytestmark = pytest.mark.gpu


def _run(w, **kw):
    r = runner(w, kv_dtype="bf16", **kw)
    r.step()
    torch.cuda.synchronize()
    return r


CASES = {
    "tiny": (lambda: wl.make("tiny"), dict(num_splits=8)),
    "ragged-h16": (lambda: wl.custom(B=4, H=16, q_len=1, seq_lens=[1, 31, 33, 517], seed=41), dict(num_splits=16)),
    "ragged-h64-rotary": (lambda: wl.custom(B=3, H=64, q_len=1, seq_lens=[700, 129, 1000], sigma_tok=1.5,
                                            rotary=True, seed=42), dict(num_splits=24)),
    "h128-two-rowgroups": (lambda: wl.custom(B=2, H=128, q_len=1, seq_lens=[300, 450], seed=43), dict(num_splits=8)),
    "mtp-causal-r256": (lambda: wl.custom(B=3, H=128, q_len=2, seq_lens=[2, 65, 257], causal=True, seed=44,
                                          n_new=2), dict(num_splits=8)),
    "mtp-causal-h32": (lambda: wl.custom(B=2, H=32, q_len=2, seq_lens=[129, 64], causal=True, seed=45, n_new=2),
                       dict(num_splits=5)),
    "more-parts-than-blocks": (lambda: wl.custom(B=2, H=16, q_len=1, seq_lens=[100, 30], seed=46),
                               dict(num_splits=64)),
    "one-part": (lambda: wl.custom(B=3, H=64, q_len=1, seq_lens=[200, 64, 333], seed=47), dict(num_splits=1)),
    "fixed-chunks": (lambda: wl.custom(B=3, H=64, q_len=1, seq_lens=[1000, 64, 129], seed=48),
                     dict(num_splits=8, kv_chunk_tokens=128)),
    "fixed-chunks-causal": (lambda: wl.custom(B=2, H=64, q_len=2, seq_lens=[513, 66], causal=True, seed=49, n_new=2),
                            dict(num_splits=3, kv_chunk_tokens=192)),
    "spread-logits": (lambda: wl.ablation(B=2, H=16, ctx=1500, seed=1320), dict(num_splits=6)),
}


@pytest.mark.parametrize("name", list(CASES))
def test_decode_bf16_matches_oracle(name):
    fac, kw = CASES[name]
    w = fac()
    print(f"[{name}] B={w.B} H={w.H} q_len={w.q_len} lens={list(map(int, w.seq_lens))} {kw}", flush=True)
    run = _run(w, **kw)
    qn, qr = w.queries()
    for b in range(w.B):
        check_sequence_bf16(run, b, reference_bf16(w, b, qn, qr), label=name)


def test_append_bf16_copies_rows():
    w = wl.custom(B=3, H=16, q_len=2, seq_lens=[70, 2, 129], causal=True, seed=51, n_new=2)
    run = _run(w, num_splits=4)
    for b in range(w.B):
        N = int(w.seq_lens[b])
        ck, kr = w.tokens(b, 0, N)
        lat, sc, rope = run.sequence_cache(b)
        assert sc is None
        assert np.array_equal(lat, ck), f"b={b}: latent rows differ"
        assert np.array_equal(rope, kr), f"b={b}: rope rows differ"


def test_empty_and_invalid_sequences_bf16():
    w = wl.custom(B=5, H=16, q_len=2, seq_lens=[0, 130, 70, 1, 64], causal=True, seed=52, n_new=0)
    run = runner(w, kv_dtype="bf16", num_splits=8)
    pt = run.page_table.clone()
    pt[1, 1] = w.num_pages + 3
    run.page_table = pt
    run.decode()
    run.combine()
    torch.cuda.synchronize()
    out = run.out.cpu().numpy()
    lse = run.lse.cpu().numpy()
    assert np.all(out[0] == 0) and np.all(lse[0] == -np.inf)
    assert np.all(np.isnan(out[1])) and np.all(np.isnan(lse[1]))
    assert np.all(np.isnan(out[3])) and np.all(np.isnan(lse[3]))
    qn, qr = w.queries()
    for b in (2, 4):
        check_sequence_bf16(run, b, reference_bf16(w, b, qn, qr), label="empty-invalid")


def test_page_shuffle_and_rerun_are_bitwise_identical_bf16():
    w1 = wl.custom(B=3, H=64, q_len=1, seq_lens=[500, 64, 1111], seed=53, shuffle_pages=False)
    w2 = wl.custom(B=3, H=64, q_len=1, seq_lens=[500, 64, 1111], seed=53, shuffle_pages=True)
    r1 = _run(w1, num_splits=12)
    r2 = _run(w2, num_splits=12)
    o1 = r1.out.clone()
    assert torch.equal(o1.view(torch.int32), r2.out.view(torch.int32))
    assert torch.equal(r1.lse.view(torch.int32), r2.lse.view(torch.int32))
    r1.decode()
    r1.combine()
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int32), r1.out.view(torch.int32))


def test_bf16_and_fp8_paths_differ_as_the_oracle_predicts():
    """The two paths on the same tokens: their difference is the FP8 quantization effect, and its
    size must match the oracle's (FP8-path oracle against the float64 BF16 reference)."""
    w = wl.custom(B=2, H=64, q_len=1, seq_lens=[900, 333], rotary=True, seed=54)
    r8 = runner(w, num_splits=8)
    r8.step()
    r16 = _run(w, num_splits=8)
    torch.cuda.synchronize()
    o8 = r8.out.cpu().numpy().astype(np.float64)
    o16 = r16.out.cpu().numpy().astype(np.float64)
    rel = np.linalg.norm(o8 - o16) / np.linalg.norm(o16)
    qn, qr = w.queries()
    num = den = 0.0
    for b in range(w.B):
        ref8, ref16 = reference(w, b, qn, qr), reference_bf16(w, b, qn, qr)
        num += float(np.sum((ref8["o"] - ref16["o"]) ** 2))
        den += float(np.sum(ref16["o"] ** 2))
    rel_oracle = np.sqrt(num / den)
    print(f"fp8 vs bf16 rel L2: device {rel:.4g}, oracle {rel_oracle:.4g}", flush=True)
    assert abs(rel - rel_oracle) <= 0.02 * rel_oracle


@pytest.mark.parametrize("name,nsample", [("headline", 3)])
def test_full_size_sampled_parity_bf16(name, nsample):
    w = wl.make(name)
    run = runner(w, kv_dtype="bf16")
    print(f"[{name} bf16] B={w.B} H={w.H} tokens={w.total_tokens} splits={run.num_splits}", flush=True)
    run.step()
    torch.cuda.synchronize()
    out = run.out.cpu().numpy()
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(run.lse.cpu().numpy()))
    qn, qr = w.queries()
    for b in sorted(set(int(round(x)) for x in np.linspace(0, w.B - 1, nsample))):
        check_sequence_bf16(run, b, reference_bf16(w, b, qn, qr), label=f"{name}-bf16")
