"""GPU: the split-KV merge with many pieces per sequence, for both slot layouts.

With one 64-row group the partials are plain rows and one wave merges one row; with several
row groups they are in accumulator tile order and a wave merges a 32 x 32 tile, its lanes
one row each with a running maximum, four pieces per round in each of the workgroup's four
waves.  Sequences here are split into tens of pieces (balanced plan with many parts, and
fixed 64-token chunks), so that every wave runs several merge rounds and the LSE pass of the
row kernel spans more than one 64-lane read; a row count that is not a multiple of 32 leaves
padding rows in the last tile.  Every row is checked against the oracle (the merge of a
sequence's pieces is its log-sum-exp over all its tokens, Algorithm 1); empty sequences give
0 / -inf and a bad page id anywhere in a many-piece sequence gives NaN rows.
"""

import numpy as np
import pytest
import torch

from paper_2602_10718_amd import workloads as wl
from gpu_common import runner, reference, check_sequence

pytestmark = pytest.mark.gpu

PLANS = {
    "balanced-many-parts": dict(num_splits=96),
    "chunks-64": dict(num_splits=90, kv_chunk_tokens=64),
}

SHAPES = {
    # (H, q_len, causal): rows 64 (one group, plain rows), 128 (two groups), 80 (two groups,
    # last 32-row tile half padding), 256 (four groups, causal)
    "r64": (64, 1, False),
    "r128": (128, 1, False),
    "r80-causal": (40, 2, True),
    "r256-causal": (128, 2, True),
}


@pytest.mark.parametrize("plan", list(PLANS))
@pytest.mark.parametrize("shape", list(SHAPES))
def test_merge_of_many_pieces_matches_oracle(shape, plan):
    H, q_len, causal = SHAPES[shape]
    w = wl.custom(B=4, H=H, q_len=q_len, seq_lens=[5000, 0, 2100, 130], causal=causal, seed=81, n_new=q_len)
    run = runner(w, **PLANS[plan])
    print(f"[combine {shape} {plan}] rows={w.rows} splits={run.num_splits} chunk={run.kv_chunk_tokens}", flush=True)
    run.out.fill_(12345.0)
    run.lse.fill_(12345.0)
    run.step()
    torch.cuda.synchronize()
    out = run.out.float().cpu().numpy()
    lse = run.lse.cpu().numpy()
    assert not np.any(out == 12345.0) and not np.any(lse == 12345.0), "a row was left unwritten"
    assert np.all(out[1] == 0) and np.all(lse[1] == -np.inf), "empty sequence"
    qn, qr = w.queries()
    for b in (0, 2, 3):
        check_sequence(run, b, reference(w, b, qn, qr), label=f"combine-{shape}-{plan}")


@pytest.mark.parametrize("shape", ["r64", "r128"])
def test_bad_page_in_a_many_piece_sequence_gives_nan_rows(shape):
    H, q_len, causal = SHAPES[shape]
    w = wl.custom(B=3, H=H, q_len=q_len, seq_lens=[4000, 900, 0], causal=causal, seed=82, n_new=0)
    run = runner(w, num_splits=80)
    pt = run.page_table.clone()
    pt[0, 37] = w.num_pages + 3                 # one bad id in the middle of sequence 0
    run.page_table = pt
    run.decode()
    run.combine()
    torch.cuda.synchronize()
    assert torch.isnan(run.out[0].float()).all() and torch.isnan(run.lse[0]).all()
    assert torch.isfinite(run.out[1].float()).all() and torch.isfinite(run.lse[1]).all()
    assert (run.out[2].float() == 0).all() and (run.lse[2] == -float("inf")).all()
    qn, qr = w.queries()
    check_sequence(run, 1, reference(w, 1, qn, qr), label=f"combine-badpage-{shape}")
