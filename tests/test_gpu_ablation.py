"""GPU: the ablation's cache quantizers (snapmla_quantize_cache_config) bit for bit against the oracle,
the decode on each configuration's cache against the oracle, and the fp32 attention reference that
bench.py --op ablation scores against."""

import numpy as np
import pytest
import torch

from oracle import granularity as gr, mla
from paper_2602_10718_amd import snapmla as sm
from paper_2602_10718_amd import workloads as wl
from gpu_common import runner, check_sequence, qk_mode
from oracle import check

pytestmark = pytest.mark.gpu


def _bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)


def _quantize_on_gpu(w, config):
    """The workload's every token through the GPU quantizer of `config`; returns the runner with the cache."""
    run = runner(w, fill=False)
    T = w.total_tokens
    cu = np.concatenate([[0], np.cumsum(w.seq_lens)]).astype(np.int32)
    ck = np.empty((T, 512), np.uint16)
    kr = np.empty((T, 64), np.uint16)
    for b in range(w.B):
        ck[cu[b]:cu[b + 1]], kr[cu[b]:cu[b + 1]] = w.tokens(b, 0, int(w.seq_lens[b]))
    scratch = torch.zeros(4, dtype=torch.int32, device="cuda")
    sm.snapmla_quantize_cache_config(_bf16(ck), _bf16(kr), run.page_table, torch.from_numpy(cu).cuda(), config,
                                     run.kv_latent, run.kv_scale, run.k_rope, scratch=scratch)
    torch.cuda.synchronize()
    return run


@pytest.mark.parametrize("config", gr.CONFIGS)
def test_quantizer_bitexact(config):
    w = wl.ablation(B=6, H=16, ctx=64)
    w.seq_lens = np.array([0, 1, 63, 64, 130, 700], np.int32)
    w = wl._finish(w)
    run = _quantize_on_gpu(w, config)
    seqs = [w.tokens(b, 0, int(w.seq_lens[b])) for b in range(w.B)]
    want = gr.quantize(config, seqs)
    lat = run.kv_latent.cpu().numpy()
    sc = run.kv_scale.cpu().numpy()
    rope = run.k_rope.view(torch.int16).cpu().numpy().view(np.uint16)
    for b in range(w.B):
        n = int(w.seq_lens[b])
        if n == 0:
            continue
        j = np.arange(n)
        pages, slots = w.page_table[b, j // 64], j % 64
        codes, sig, rb = want[b]
        assert np.array_equal(lat[pages, slots], codes), f"{config} b={b}: codes"
        assert np.array_equal(sc[pages, slots].view(np.uint32), sig.view(np.uint32)), f"{config} b={b}: scales"
        assert np.array_equal(rope[pages, slots], rb), f"{config} b={b}: rope"


@pytest.mark.parametrize("config", gr.CONFIGS)
def test_decode_on_config_cache(config):
    w = wl.ablation(B=3, H=16, ctx=64)
    w.seq_lens = np.array([900, 64, 1300], np.int32)
    w = wl._finish(w)
    run = _quantize_on_gpu(w, config)
    run.decode()
    run.combine()
    torch.cuda.synchronize()
    qn, qr = w.queries()
    seqs = [w.tokens(b, 0, int(w.seq_lens[b])) for b in range(w.B)]
    caches = gr.quantize(config, seqs)
    for b in range(w.B):
        ck, kr = seqs[b]
        ref = check.sequence_reference(qn[b], qr[b], ck, kr, w.tau, w.q_len, w.H, w.causal, cache=caches[b],
                                       qk=qk_mode(run))
        check_sequence(run, b, ref, label=f"abl-{config}")


def test_torch_reference_matches_oracle():
    import bench
    w = wl.ablation(B=2, H=8, ctx=700)
    qn, qr = w.queries()
    for b in range(w.B):
        ck, kr = w.tokens(b, 0, 700)
        vis = np.full(w.H, 700)
        got = bench.torch_attention_f32(_bf16(qn[b].reshape(-1, 512)), _bf16(qr[b].reshape(-1, 64)), _bf16(ck),
                                        _bf16(kr), w.tau, vis).double().cpu().numpy()
        want = mla.bf16_reference(qn[b].reshape(-1, 512), qr[b].reshape(-1, 64), ck, kr, w.tau, vis)[0]
        assert np.max(np.abs(got - want)) <= 1e-4 * np.max(np.abs(want))
