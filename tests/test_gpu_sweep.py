"""GPU: every (H, q_len) of the sensitivity sweep against the oracle.

Small sequences for all eight shapes in the launch configuration bench.py
--op sweep uses (the default split plan of each shape), and sampled sequences
of the full sweep workload (batch 32, lengths U[16K, 128K]) for the smallest
and the largest row count.
"""

import numpy as np
import pytest
import torch

from paper_2602_10718_amd import workloads as wl
from gpu_common import runner, reference, check_sequence

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("q_len", wl.SWEEP_QLEN)
@pytest.mark.parametrize("H", wl.SWEEP_HEADS)
def test_sweep_shape_small(H, q_len):
    w = wl.custom(B=3, H=H, q_len=q_len, seq_lens=[1100, 64 + q_len, 2049], causal=q_len == 2, n_new=q_len,
                  sigma_tok=1.5, rotary=True, seed=300 + H + q_len)
    run = runner(w)
    print(f"[sweep-small H={H} q_len={q_len}] splits={run.num_splits}", flush=True)
    run.step()
    torch.cuda.synchronize()
    qn, qr = w.queries()
    for b in range(w.B):
        check_sequence(run, b, reference(w, b, qn, qr), label=f"H{H}q{q_len}")


@pytest.fixture(scope="module")
def sweep_cache():
    w = wl.sweep(16, 1)
    r = runner(w)
    return r.kv_latent, r.kv_scale, r.k_rope


@pytest.mark.parametrize("H,q_len", [(16, 1), (128, 2)])
def test_sweep_full_size_sampled(sweep_cache, H, q_len):
    w = wl.sweep(H, q_len)
    run = runner(w, cache=sweep_cache)
    print(f"[sweep-full H={H} q_len={q_len}] tokens={w.total_tokens} splits={run.num_splits}", flush=True)
    run.step()
    torch.cuda.synchronize()
    out = run.out.float().cpu().numpy()
    assert np.all(np.isfinite(out))
    qn, qr = w.queries()
    for b in (int(np.argmin(w.seq_lens)), int(np.argsort(w.seq_lens)[w.B // 2])):
        check_sequence(run, b, reference(w, b, qn, qr), label=f"sweep H{H}q{q_len}")
