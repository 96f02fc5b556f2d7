"""GPU: spread attention over thousands of tokens, where the P quantization shapes the output.

On the named workloads' data the attention of most rows rests on a few tokens, so the block
quantization of the probabilities (Section 3.2 (i)-(ii)) and the Appendix D bookkeeping that
undoes it barely move the output.  Here the content logits are shrunk (q_nope x 0.05, per-token
magnitudes lognormal(0, 0.3), no outlier channels), so every row spreads its weight over
hundreds of tokens (largest weight ~0.002) and dropping the P quantization moves the output by
a relative L2 of ~2 %.  Each case first shows that sensitivity on the oracle -- its unquantized-P
form (mla.decode_none) falls outside the derived bound on a good fraction of the elements -- and
then requires the device output of every sequence inside that bound and the benchmark spec
tolerance, in both QK modes, for the three kernel schedules: one 64-row group, the causal MTP
rows, and two row groups (the several-row-group schedule), each over a plan with short ranges
(many pieces per sequence) and one with long ranges (many blocks per workgroup).
"""

import numpy as np
import pytest
import torch

from oracle import check, mla
from paper_2602_10718_amd import workloads as wl
from gpu_common import runner, reference, check_sequence

pytestmark = pytest.mark.gpu

CASES = {
    # name: (H, q_len, causal, seq_lens)
    "h64": (64, 1, False, [4096 + 37, 9000, 2500, 6143, 1281]),
    "mtp_causal": (32, 2, True, [5000, 64 * 37, 3001]),
    "two_groups": (128, 1, False, [4100, 2049, 3333]),
}


def _workload(H, q_len, causal, lens, seed):
    w = wl.custom(B=len(lens), H=H, q_len=q_len, seq_lens=lens, causal=causal, sigma_tok=0.3, seed=seed)
    w.outlier_gain = 1.0
    w.q_nope_scale = 0.05
    return w


@pytest.mark.parametrize("num_splits", [None, 16])
@pytest.mark.parametrize("qk", ["mfma8", "exact"])
@pytest.mark.parametrize("name", list(CASES))
def test_spread_attention_matches_oracle(name, qk, num_splits):
    H, q_len, causal, lens = CASES[name]
    w = _workload(H, q_len, causal, lens, seed=61 + len(name))
    run = runner(w, num_splits=num_splits, out_dtype=torch.float32, exact_qk=(qk == "exact"))
    print(f"[spread {name} {qk}] B={w.B} rows={w.rows} tokens={w.total_tokens} splits={run.num_splits}",
          flush=True)
    run.step()
    torch.cuda.synchronize()
    qn, qr = w.queries()
    for b in range(w.B):
        ref = reference(w, b, qn, qr, qk=qk)
        # the case is sensitive to the P quantization: without it the output leaves the bound
        ob, _, _ = check.bounds(ref)
        o_none, _ = mla.decode_none(ref["q8"], ref["sq"], ref["qr"], ref["c8"], ref["sk"], ref["kr"], ref["tau"],
                                    ref["vis"], qk=qk)
        outside = float(np.mean(np.abs(o_none - ref["o"]) > ob))
        assert outside > 0.01, f"{name} b={b}: unquantized P stays inside the bound ({outside:.3g})"
        wmax = float(np.max(ref["parts"]["e"] / ref["parts"]["lam"][:, None]))
        assert wmax < 0.05, f"{name} b={b}: attention not spread (largest weight {wmax:.3g})"
        m = check_sequence(run, b, ref, label=f"spread-{name}")
        assert m["rel_l2"] < 1e-3, f"{name} b={b}: rel-L2 {m['rel_l2']:.3g} on spread attention"
