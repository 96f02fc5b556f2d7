"""GPU: the decode's direct rows -- sequences that one piece covers finalised by the decode itself.

A piece that holds a whole sequence ends with o = O / l and LSE = m + ln(sigma_P l) (Algorithm 1
finalisation) written straight into out/lse; the merge of a single piece is exact (weight
exp(0) = 1, one term), so the direct rows must equal, bit for bit, what the partial + combine
path gives.  Checked for plans that mix one-piece and split sequences, for both cache types, both
output types and one and two row groups.  The unsplit plan (fixed chunks as long as the page table,
one split) needs no combine at all when the decode writes direct rows (the FP8-cache decode with one
64-row group, the BF16-cache decode always): every row, including those of empty sequences (0, -inf)
and of sequences a data error rejects (NaN), comes from the decode call and matches the oracle.
With several row groups the FP8-cache decode writes partials only and the combine writes the rows.
"""

import numpy as np
import pytest
import torch

from paper_2602_10718_amd import workloads as wl
from gpu_common import runner, reference, check_sequence

pytestmark = pytest.mark.gpu


def _bits(t):
    t = t.contiguous()
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).cpu().numpy()


PLANS = {
    # balanced plan with few parts: short sequences fall inside one part, long ones span several
    "balanced": dict(num_splits=4),
    # fixed chunks: sequences up to one chunk are one piece
    "chunks": dict(num_splits=8, kv_chunk_tokens=256),
    # one piece per sequence
    "unsplit": dict(unsplit=True),
}


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("kv_dtype", ["e4m3", "bf16"])
@pytest.mark.parametrize("H", [64, 128])
@pytest.mark.parametrize("plan", list(PLANS))
def test_direct_rows_equal_partial_and_combine_bitwise(plan, H, kv_dtype, out_dtype):
    w = wl.custom(B=6, H=H, q_len=1, seq_lens=[64, 1200, 0, 190, 700, 33], seed=71)
    ref_run = runner(w, out_dtype=out_dtype, kv_dtype=kv_dtype, direct=False, **PLANS[plan])
    run = runner(w, out_dtype=out_dtype, kv_dtype=kv_dtype, cache=(ref_run.kv_latent, ref_run.kv_scale,
                                                                   ref_run.k_rope), **PLANS[plan])
    print(f"[direct {plan} H={H} {kv_dtype} {out_dtype}] splits={run.num_splits} chunk={run.kv_chunk_tokens} "
          f"needs_combine={run.needs_combine}", flush=True)
    ref_run.decode()
    ref_run.combine()
    run.out.fill_(7.0)
    run.lse.fill_(7.0)
    run.decode()
    run.combine()
    torch.cuda.synchronize()
    assert np.array_equal(_bits(run.out), _bits(ref_run.out)), "direct rows differ from partial + combine"
    assert np.array_equal(_bits(run.lse), _bits(ref_run.lse)), "direct LSEs differ from partial + combine"


@pytest.mark.parametrize("qk", ["mfma8", "exact"])
@pytest.mark.parametrize("H,q_len,causal", [(64, 1, False), (32, 2, True), (128, 1, False)])
def test_unsplit_plan_without_combine_matches_oracle(H, q_len, causal, qk):
    w = wl.custom(B=5, H=H, q_len=q_len, seq_lens=[900, 0, 64, 1, 2100], causal=causal, seed=72, n_new=q_len)
    run = runner(w, unsplit=True, exact_qk=(qk == "exact"))
    assert run.needs_combine == (w.rows > 64)
    run.out.fill_(12345.0)
    run.lse.fill_(12345.0)
    run.step()                              # append + decode (and the combine only with several row groups)
    torch.cuda.synchronize()
    out = run.out.cpu().numpy()
    lse = run.lse.cpu().numpy()
    assert not np.any(out == 12345.0) and not np.any(lse == 12345.0), "a row was left unwritten"
    assert np.all(out[1] == 0) and np.all(lse[1] == -np.inf), "empty sequence"
    if q_len == 2:                          # 0 < seq_len < q_len: rejected
        assert np.all(np.isnan(out[3])) and np.all(np.isnan(lse[3]))
    qn, qr = w.queries()
    for b in range(w.B):
        if int(w.seq_lens[b]) >= q_len:
            check_sequence(run, b, reference(w, b, qn, qr, qk=qk), label=f"unsplit-H{H}")
    # a rejected sequence (longer than the page table) and a bad page id: NaN rows from the decode alone
    seq = run.seq_lens.clone()
    seq[0] = 64 * w.max_pages + 1
    run.seq_lens = seq
    pt = run.page_table.clone()
    pt[4, 3] = w.num_pages + 5
    run.page_table = pt
    run.out.fill_(12345.0)
    run.decode()
    if run.needs_combine:
        run.combine()
    torch.cuda.synchronize()
    assert torch.isnan(run.out[0]).all() and torch.isnan(run.lse[0]).all()
    assert torch.isnan(run.out[4]).all() and torch.isnan(run.lse[4]).all()
    assert torch.isfinite(run.out[2]).all()
    # combine after the unsplit decode leaves every row as it is
    before = _bits(run.out), _bits(run.lse)
    run.combine()
    torch.cuda.synchronize()
    assert np.array_equal(_bits(run.out), before[0]) and np.array_equal(_bits(run.lse), before[1])
