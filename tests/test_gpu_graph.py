"""GPU: a decode step captured as a HIP graph gives, on every replay, the eager result bit for bit."""

import numpy as np
import pytest
import torch

from paper_2602_10718_amd import workloads as wl
from gpu_common import runner

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("kw", [dict(num_splits=16), dict(num_splits=6, kv_chunk_tokens=128)])
def test_graph_replay_matches_eager(kw):
    w = wl.custom(B=3, H=64, q_len=1, seq_lens=[900, 64, 1500], seed=41)
    run = runner(w, out_dtype=torch.float32, **kw)
    run.step()
    torch.cuda.synchronize()
    ref_o = run.out.clone()
    ref_l = run.lse.clone()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run.step()
    for k in range(3):
        run.out.fill_(float("nan"))
        run.lse.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(run.out.view(torch.int32), ref_o.view(torch.int32)), f"replay {k}"
        assert torch.equal(run.lse.view(torch.int32), ref_l.view(torch.int32)), f"replay {k}"
        run.step()                      # eager work between the replays
        torch.cuda.synchronize()
        assert np.array_equal(run.out.cpu().numpy().view(np.int32), ref_o.cpu().numpy().view(np.int32))
