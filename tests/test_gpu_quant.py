"""GPU: the E4M3 conversion and the per-token quantizers must match the oracle bit for bit."""

import numpy as np
import pytest
import torch

from oracle import e4m3, quant
from paper_2602_10718_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sm():
    from paper_2602_10718_amd import snapmla
    return snapmla


def test_e4m3_encode_every_float32_below_464(sm):
    """All float32 patterns with |x| < 464 (both signs) against the oracle's rounding thresholds."""
    th = torch.from_numpy(e4m3.fp32_thresholds().astype(np.int64)).cuda()
    top = int(np.array([464.0], np.float32).view(np.uint32)[0])
    chunk = 1 << 27
    bad = 0
    for start in range(0, top, chunk):
        end = min(top, start + chunk)
        pats = torch.arange(start, end, dtype=torch.int64, device="cuda")
        x = pats.to(torch.int32).view(torch.float32)
        codes = torch.empty(end - start, dtype=torch.uint8, device="cuda")
        sm.snapmla_e4m3_encode(x, codes)
        expect = torch.searchsorted(th, pats, right=True)
        bad += int((codes.to(torch.int64) != expect).sum())
        sm.snapmla_e4m3_encode(-x, codes)      # negative values: same magnitude code with the sign bit
        bad += int((codes.to(torch.int64) != (expect | 0x80)).sum())
    assert bad == 0


def test_e4m3_encode_saturates(sm):
    x = torch.tensor([448.0, 463.99, 464.0, 500.0, 1e30, -1e30, 0.0, -0.0], device="cuda")
    c = torch.empty(8, dtype=torch.uint8, device="cuda")
    sm.snapmla_e4m3_encode(x, c)
    assert c.cpu().tolist() == [0x7E, 0x7E, 0x7E, 0x7E, 0x7E, 0xFE, 0x00, 0x80]


def _bits_to_dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


@pytest.mark.parametrize("sigma", [0.0, 1.0, 3.0])
def test_quantize_rows_bitexact(sm, sigma):
    rng = np.random.default_rng(7)
    n = 4099
    x = rng.standard_normal((n, 512)).astype(np.float32)
    x *= np.exp(rng.standard_normal(n) * sigma).astype(np.float32)[:, None]
    x[:, [1, 100, 200, 511]] *= 20
    x[5] = 0.0
    x[6, 3] = 1e-30
    x[7] *= np.float32(1e-12)
    bits = wl.f32_to_bf16_bits(x)
    codes = torch.empty((n, 512), dtype=torch.uint8, device="cuda")
    scale = torch.empty(n, dtype=torch.float32, device="cuda")
    sm.snapmla_quantize_rows(_bits_to_dev(bits), codes, scale)
    c_ref, s_ref = quant.quantize_rows(bits)
    assert np.array_equal(scale.cpu().numpy().view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(codes.cpu().numpy(), c_ref)


def test_quantize_append_paged_bitexact(sm):
    """Bulk fill + per-step append into shuffled pages; every slot equals the oracle, untouched slots stay."""
    w = wl.custom(B=3, H=16, q_len=1, seq_lens=[1, 130, 700], sigma_tok=1.5, rotary=True, seed=11, n_new=2)
    from paper_2602_10718_amd.runner import DecodeRunner
    run = DecodeRunner(w, num_splits=8)
    run.append()
    torch.cuda.synchronize()
    for b in range(w.B):
        N = int(w.seq_lens[b])
        ck, kr = w.tokens(b, 0, N)
        c_ref, s_ref = quant.quantize_rows(ck)
        codes, scales, rope = run.sequence_cache(b)
        assert np.array_equal(codes, c_ref), f"seq {b}"
        assert np.array_equal(scales.view(np.uint32), s_ref.view(np.uint32)), f"seq {b}"
        assert np.array_equal(rope, kr), f"seq {b}"
    # slots past each sequence end were never written (still zero)
    for b in range(w.B):
        N = int(w.seq_lens[b])
        last = w.page_table[b, (N - 1) // 64]
        tail = run.kv_latent[int(last), N % 64:].cpu().numpy() if N % 64 else np.zeros(0)
        assert np.all(tail == 0)


def test_quantize_append_skips_invalid_slots(sm):
    w = wl.custom(B=2, H=16, q_len=1, seq_lens=[64, 64], seed=12, n_new=1)
    from paper_2602_10718_amd.runner import DecodeRunner
    run = DecodeRunner(w, num_splits=8, fill=False)
    pt = run.page_table.clone()
    pt[0, 0] = w.num_pages + 5           # out of range: must be skipped
    seq = torch.tensor([64, 10_000], dtype=torch.int32, device="cuda")   # beyond max_pages*64: skipped
    before = run.kv_latent.clone()
    sm.snapmla_quantize_append(run.new_ckv, run.new_krope, pt, seq, w.num_pages, run.kv_latent, run.kv_scale,
                               run.k_rope)
    torch.cuda.synchronize()
    assert torch.equal(before, run.kv_latent)
