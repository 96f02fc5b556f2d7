"""GPU: decode + combine against the oracle, edge cases, bitwise invariances."""

import math

import numpy as np
import pytest
import torch

from paper_2602_10718_amd import workloads as wl
from gpu_common import runner, reference, check_sequence

pytestmark = pytest.mark.gpu


def _run(w, **kw):
    r = runner(w, **kw)
    r.step()
    torch.cuda.synchronize()
    return r


CASES = {
    # name: (workload factory, runner kwargs)
    "tiny": (lambda: wl.make("tiny"), dict(num_splits=8)),
    "ragged-h16": (lambda: wl.custom(B=4, H=16, q_len=1, seq_lens=[1, 63, 64, 517], seed=21), dict(num_splits=16)),
    "ragged-h64-rotary": (lambda: wl.custom(B=3, H=64, q_len=1, seq_lens=[700, 129, 1000], sigma_tok=1.5,
                                            rotary=True, seed=22), dict(num_splits=24)),
    "h128-two-rowgroups": (lambda: wl.custom(B=2, H=128, q_len=1, seq_lens=[300, 450], seed=23), dict(num_splits=8)),
    "mtp-causal-r256": (lambda: wl.custom(B=3, H=128, q_len=2, seq_lens=[2, 65, 257], causal=True, seed=24,
                                          n_new=2), dict(num_splits=8)),
    "mtp-causal-h32": (lambda: wl.custom(B=2, H=32, q_len=2, seq_lens=[129, 64], causal=True, seed=25, n_new=2),
                       dict(num_splits=5)),
    "more-parts-than-blocks": (lambda: wl.custom(B=2, H=16, q_len=1, seq_lens=[100, 30], seed=26),
                               dict(num_splits=64)),
    "one-part": (lambda: wl.custom(B=3, H=64, q_len=1, seq_lens=[200, 64, 333], seed=27), dict(num_splits=1)),
    "fixed-chunks": (lambda: wl.custom(B=3, H=64, q_len=1, seq_lens=[1000, 64, 129], seed=28),
                     dict(num_splits=8, kv_chunk_tokens=128)),
    "fixed-chunks-causal": (lambda: wl.custom(B=2, H=64, q_len=2, seq_lens=[513, 66], causal=True, seed=29, n_new=2),
                            dict(num_splits=3, kv_chunk_tokens=192)),
}


@pytest.mark.parametrize("qk", ["mfma8", "exact"])
@pytest.mark.parametrize("name", list(CASES))
def test_decode_matches_oracle(name, qk):
    """Both QK modes: the default decode (content term on the FP8 matrix cores) against the oracle
    that forms the content term the same way, the SNAPMLA_DECODE_EXACT_QK decode against the exact
    oracle; each within the derived bounds and the benchmark spec tolerance."""
    fac, kw = CASES[name]
    w = fac()
    run = _run(w, exact_qk=(qk == "exact"), **kw)
    qn, qr = w.queries()
    for b in range(w.B):
        ref = reference(w, b, qn, qr, qk=qk)
        check_sequence(run, b, ref, label=name)


def test_tame_data_tight_agreement():
    """Small logits: the derived bounds shrink to ~1e-4 and the output must follow them."""
    w = wl.custom(B=2, H=64, q_len=1, seq_lens=[777, 300], sigma_tok=0.2, seed=31)
    run = _run(w, num_splits=16)
    qn, qr = w.queries()
    qn = wl.f32_to_bf16_bits(wl.bf16_bits_to_f32(qn) * np.float32(0.05))   # shrink the content logits
    run.q_nope.copy_(torch.from_numpy(qn.view(np.int16)).cuda().view(torch.bfloat16))
    run.decode()
    run.combine()
    torch.cuda.synchronize()
    for b in range(w.B):
        m = check_sequence(run, b, reference(w, b, qn, qr), label="tame")
        assert m["rel_l2"] < 2e-3 and m["lse_max_abs"] < 1e-3


def test_empty_and_invalid_sequences():
    w = wl.custom(B=5, H=16, q_len=2, seq_lens=[0, 130, 70, 1, 64], causal=True, seed=32, n_new=0)
    run = runner(w, num_splits=8)
    # sequence 1: a page id out of range -> NaN rows; sequence 3 has 0 < seq_len < q_len -> NaN
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
        check_sequence(run, b, reference(w, b, qn, qr), label="empty-invalid")
    # a sequence longer than max_pages * 64 is rejected
    seq = run.seq_lens.clone()
    seq[2] = 64 * w.max_pages + 1
    run.seq_lens = seq
    run.decode()
    run.combine()
    torch.cuda.synchronize()
    assert np.all(np.isnan(run.out[2].cpu().numpy()))
    assert np.isfinite(run.out[4].cpu().numpy()).all()


def test_page_shuffle_and_rerun_are_bitwise_identical():
    w1 = wl.custom(B=3, H=64, q_len=1, seq_lens=[500, 64, 1111], seed=33, shuffle_pages=False)
    w2 = wl.custom(B=3, H=64, q_len=1, seq_lens=[500, 64, 1111], seed=33, shuffle_pages=True)
    assert not np.array_equal(w1.page_table, w2.page_table)
    r1 = _run(w1, num_splits=12)
    r2 = _run(w2, num_splits=12)
    o1 = r1.out.clone()
    assert torch.equal(o1.view(torch.int32), r2.out.view(torch.int32))
    assert torch.equal(r1.lse.view(torch.int32), r2.lse.view(torch.int32))
    r1.decode()
    r1.combine()
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int32), r1.out.view(torch.int32))


def test_split_plans_agree():
    """Different split plans give the same result up to float32 merge rounding."""
    w = wl.custom(B=3, H=64, q_len=1, seq_lens=[2000, 640, 3001], seed=34)
    outs = []
    for kw in (dict(num_splits=1), dict(num_splits=7), dict(num_splits=40), dict(num_splits=50, kv_chunk_tokens=64)):
        r = _run(w, **kw)
        outs.append((r.out.cpu().numpy().astype(np.float64), r.lse.cpu().numpy().astype(np.float64)))
    o0, l0 = outs[0]
    for o, l in outs[1:]:
        assert np.linalg.norm(o - o0) / np.linalg.norm(o0) < 1e-5
        assert np.max(np.abs(l - l0)) < 1e-4


def test_bf16_output():
    w = wl.custom(B=2, H=16, q_len=1, seq_lens=[300, 100], seed=35)
    r32 = _run(w, num_splits=8)
    r16 = _run(w, num_splits=8, out_dtype=torch.bfloat16)
    assert torch.equal(r32.out.to(torch.bfloat16).view(torch.int16), r16.out.view(torch.int16))


def test_plan_with_many_sequences_and_units():
    """Split plans whose start descriptors take the prep kernel's general paths: more
    sequences than scan threads (B = 300, the prefix read back from global memory) and
    more units than threads (fixed chunks: 300 sequences x 2 chunks)."""
    rng = np.random.default_rng(36)
    lens = rng.integers(1, 260, 300).astype(np.int32)
    lens[[5, 77, 150]] = 0                                  # empty sequences inside the range
    w = wl.custom(B=300, H=16, q_len=1, seq_lens=lens.tolist(), seed=36)
    qn, qr = w.queries()
    for kw in (dict(num_splits=40), dict(num_splits=2, kv_chunk_tokens=192)):
        run = _run(w, **kw)
        out = run.out.cpu().numpy()
        assert np.all(np.isfinite(out)), f"{kw}: non-finite output"
        lse = run.lse.cpu().numpy()
        for b in (5, 77, 150):                              # empty: output 0, LSE -inf
            assert np.all(out[b] == 0) and np.all(lse[b] == -np.inf)
        for b in (0, 1, 4, 6, 76, 78, 149, 151, 255, 256, 257, 299):
            check_sequence(run, b, reference(w, b, qn, qr), label=f"many-seq {kw}")


@pytest.mark.parametrize("name", ["ragged-h16", "h128-two-rowgroups", "fixed-chunks-causal"])
def test_decode_kernel_alone_repeats_the_decode_launch(name):
    """snapmla_debug_decode_kernel, the decode launch alone that bench.py times for the roofline, over the
    workspace a snapmla_decode call prepared: after it and the combine, every output row and LSE equals the
    full call's bit for bit (direct rows included: the outputs are overwritten with a marker in between)."""
    fac, kw = CASES[name]
    w = fac()
    run = runner(w, **kw)
    print(f"[decode kernel alone] {name}", flush=True)
    run.decode()
    run.combine()
    torch.cuda.synchronize()
    out1, lse1 = run.out.clone(), run.lse.clone()
    run.out.fill_(12345.0)
    run.lse.fill_(12345.0)
    run.decode_kernel_only()
    run.combine()
    torch.cuda.synchronize()
    assert torch.equal(run.out.view(torch.int32), out1.view(torch.int32))
    assert torch.equal(run.lse.view(torch.int32), lse1.view(torch.int32))


def test_decode_kernel_alone_needs_a_matching_preparation():
    """The decode launch alone is refused for a workspace that no FP8 decode call prepared, or that one
    with other sizes prepared last, and accepted again once a matching call has prepared it."""
    fac, kw = CASES["ragged-h16"]
    w = fac()
    from paper_2602_10718_amd import snapmla as sm
    run = runner(w, **kw)
    print("[decode kernel alone: preparation check]", flush=True)
    run.decode()
    run.combine()
    torch.cuda.synchronize()
    out1 = run.out.clone()
    fresh = torch.zeros_like(run.workspace)
    with pytest.raises(RuntimeError, match="not prepared"):
        sm.snapmla_debug_decode_kernel(run.q_nope, run.q_rope, run.kv_latent, run.kv_scale, run.k_rope,
                                       run.page_table, run.seq_lens, w.tau, w.causal, run.num_splits,
                                       run.kv_chunk_tokens, fresh)
    with pytest.raises(RuntimeError, match="not prepared"):
        sm.snapmla_debug_decode_kernel(run.q_nope, run.q_rope, run.kv_latent, run.kv_scale, run.k_rope,
                                       run.page_table, run.seq_lens, w.tau, w.causal, run.num_splits // 2,
                                       run.kv_chunk_tokens, run.workspace)
    run.out.fill_(12345.0)
    run.decode_kernel_only()
    run.combine()
    torch.cuda.synchronize()
    assert torch.equal(run.out.view(torch.int32), out1.view(torch.int32))


@pytest.mark.parametrize("splits", [600, 1024, 1500])
def test_padded_plan_with_more_parts_than_positions(splits):
    """The balanced plan of a one-row-group launch charges each sequence start 4 virtual
    blocks.  With short sequences and many parts, most parts fall inside those charges and
    get no blocks; 600 and 1,024 parts take the prep kernel's unit table, 1,500 its binary
    searches.  Every sequence must still come out whole: empty ones 0 / -inf, the others
    equal to the oracle."""
    rng = np.random.default_rng(37)
    lens = rng.integers(1, 200, 200).astype(np.int32)
    lens[[3, 64, 65, 199]] = 0                              # empty sequences, one of them last
    w = wl.custom(B=200, H=16, q_len=1, seq_lens=lens.tolist(), seed=37)
    qn, qr = w.queries()
    run = _run(w, num_splits=splits)
    print(f"[padded plan] splits={splits} blocks={int(((lens + 63) // 64).sum())}", flush=True)
    out = run.out.cpu().numpy()
    lse = run.lse.cpu().numpy()
    assert np.all(np.isfinite(out)), "non-finite output"
    for b in (3, 64, 65, 199):
        assert np.all(out[b] == 0) and np.all(lse[b] == -np.inf)
    for b in (0, 1, 2, 4, 63, 66, 100, 150, 197, 198):
        check_sequence(run, b, reference(w, b, qn, qr), label=f"padded plan {splits}")


@pytest.mark.parametrize("name", ["ragged-h16", "h128-two-rowgroups", "mtp-causal-r256", "fixed-chunks-causal"])
def test_append_decode_equals_separate_calls(name):
    """snapmla_append_decode (append inside the preparation launch) against snapmla_quantize_append
    followed by snapmla_decode: the same cache bytes, outputs and LSEs, bit for bit."""
    fac, kw = CASES[name]
    w = fac()
    fused, split = runner(w, **kw), runner(w, **kw)
    print(f"[append_decode] {name}", flush=True)
    fused.append_decode()
    fused.combine()
    split.append()
    split.decode()
    split.combine()
    torch.cuda.synchronize()
    for a, b in ((fused.kv_latent, split.kv_latent), (fused.kv_scale, split.kv_scale), (fused.k_rope, split.k_rope)):
        assert torch.equal(a.view(torch.uint8), b.view(torch.uint8))
    assert torch.equal(fused.out.view(torch.int32), split.out.view(torch.int32))
    assert torch.equal(fused.lse.view(torch.int32), split.lse.view(torch.int32))


def test_append_decode_data_errors_and_no_append_equal_separate_calls():
    """The fused call on data errors (an out-of-range page id under the new tokens, an empty
    sequence, 0 < seq_len < q_len) and with n_new = 0 matches the separate calls bit for bit."""
    w = wl.custom(B=5, H=16, q_len=2, seq_lens=[0, 130, 70, 1, 64], causal=True, seed=34, n_new=2)
    fused, split = runner(w, num_splits=8), runner(w, num_splits=8)
    for r in (fused, split):
        pt = r.page_table.clone()
        pt[1, 2] = w.num_pages + 3            # the page of sequence 1's new tokens
        r.page_table = pt
    print("[append_decode] data errors", flush=True)
    fused.append_decode()
    fused.combine()
    split.append()
    split.decode()
    split.combine()
    torch.cuda.synchronize()
    for a, b in ((fused.kv_latent, split.kv_latent), (fused.kv_scale, split.kv_scale), (fused.k_rope, split.k_rope)):
        assert torch.equal(a.view(torch.uint8), b.view(torch.uint8))
    assert torch.equal(fused.out.view(torch.int32), split.out.view(torch.int32))
    assert torch.equal(fused.lse.view(torch.int32), split.lse.view(torch.int32))
    assert np.all(np.isnan(fused.out[1].float().cpu().numpy()))

    w0 = wl.custom(B=3, H=64, q_len=1, seq_lens=[300, 64, 129], seed=35, n_new=0)
    fused, split = runner(w0, num_splits=8), runner(w0, num_splits=8)
    assert fused.new_ckv.shape[1] == 0
    print("[append_decode] n_new = 0", flush=True)
    fused.append_decode()
    fused.combine()
    split.decode()
    split.combine()
    torch.cuda.synchronize()
    assert torch.equal(fused.out.view(torch.int32), split.out.view(torch.int32))
    assert torch.equal(fused.lse.view(torch.int32), split.lse.view(torch.int32))


@pytest.mark.parametrize("kv_dtype", ["e4m3", "bf16"])
def test_handshake_wait_that_gives_up_marks_the_piece_nan(kv_dtype):
    """A bounded handshake wait that reaches its limit must not let stale codes through silently:
    with the limit set to 0 polls (a host-side setting; every kernel still runs to completion)
    every piece is marked and every output and LSE comes out NaN; with the default limit the
    same runner is back to the oracle's results."""
    from paper_2602_10718_amd import snapmla as sm
    w = wl.custom(B=2, H=64, q_len=1, seq_lens=[300, 200], seed=41)
    run = runner(w, num_splits=4, kv_dtype=kv_dtype)
    try:
        sm.snapmla_debug_set_spin_limit(0)
        run.step()
        torch.cuda.synchronize()
        assert torch.isnan(run.out).all() and torch.isnan(run.lse).all()
    finally:
        sm.snapmla_debug_set_spin_limit(1 << 22)
    run.decode()
    run.combine()
    torch.cuda.synchronize()
    assert torch.isfinite(run.out).all() and torch.isfinite(run.lse).all()
    if kv_dtype == "e4m3":
        qn, qr = w.queries()
        for b in range(w.B):
            check_sequence(run, b, reference(w, b, qn, qr), label="after-give-up")

