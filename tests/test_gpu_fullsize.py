"""GPU: full-size workloads in the launch configuration bench.py times, checked on sampled sequences.

Configs 2-5 are built at their full sizes (the whole paged cache through
snapmla_quantize_append, the default split plan of bench.py).  The oracle is
evaluated for a sample of sequences (first, middle, last; eight for the MTP
config) and every sampled output and LSE must lie inside the derived bounds
and the benchmark spec tolerance, in both QK modes (each against the oracle in the
same mode).  The rest of the batch is checked through properties
that hold at any size: finite outputs and LSEs, and the appended tokens'
cache bytes equal to the oracle quantizer's.
"""

import numpy as np
import pytest
import torch

from oracle import quant
from paper_2602_10718_amd import workloads as wl
from gpu_common import runner, reference, check_sequence

pytestmark = pytest.mark.gpu


def _sample(B, n):
    if n >= B:
        return list(range(B))
    return sorted(set(int(round(x)) for x in np.linspace(0, B - 1, n)))


@pytest.mark.parametrize("qk", ["mfma8", "exact"])
@pytest.mark.parametrize("name,nsample", [("dsv3", 3), ("headline", 3), ("longsplit", 2), ("mtp", 8)])
def test_full_size_sampled_parity(name, nsample, qk):
    w = wl.make(name)
    run = runner(w, out_dtype=torch.float32, exact_qk=(qk == "exact"))
    print(f"[{name}] B={w.B} H={w.H} q_len={w.q_len} tokens={w.total_tokens} splits={run.num_splits} "
          f"chunk={run.kv_chunk_tokens}", flush=True)
    run.step()
    torch.cuda.synchronize()
    out = run.out.cpu().numpy()
    lse = run.lse.cpu().numpy()
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse)), f"{name}: non-finite output"
    qn, qr = w.queries()
    for b in _sample(w.B, nsample):
        check_sequence(run, b, reference(w, b, qn, qr, qk=qk), label=name)
    # the tokens appended by the step landed bit-exactly in their pages
    for b in _sample(w.B, 4):
        N = int(w.seq_lens[b])
        lo = max(0, N - w.n_new)
        ck, kr = w.tokens(b, lo, N)
        codes, scales = quant.quantize_rows(ck)
        c_dev, s_dev, r_dev = run.sequence_cache(b)
        assert np.array_equal(c_dev[lo:N], codes), f"{name} b={b}: appended codes differ"
        assert np.array_equal(s_dev[lo:N].view(np.uint32), scales.view(np.uint32)), f"{name} b={b}: scales"
        assert np.array_equal(r_dev[lo:N], kr), f"{name} b={b}: rope bits"
