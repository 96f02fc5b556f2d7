"""GPU: snapmla_fetch_dequant against the oracle, bit for bit (oracle/fetch.py).

The output is a deterministic function of the cache bytes (one float32
product, one bf16 rounding), so every output bit is compared.  Cases: ragged
lengths (0, 1, a partial page, whole pages) through a shuffled page table;
every E4M3 code; both data errors; a cache written by snapmla_quantize_append;
and sampled sequences of the headline cache in the launch configuration that
bench.py --op fetch_dequant times.
"""

import numpy as np
import pytest
import torch

from oracle import fetch
from paper_2602_10718_amd import snapmla as sm
from paper_2602_10718_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _u16_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)


def _run(lat, sc, rope, pt, cu, num_pages=None):
    lat_d = torch.from_numpy(lat).cuda()
    sc_d = torch.from_numpy(sc).cuda()
    rope_d = _u16_dev(rope)
    pt_d = torch.from_numpy(pt.astype(np.int32)).cuda()
    cu_d = torch.from_numpy(cu.astype(np.int32)).cuda()
    out = torch.full((int(cu[-1]), 576), -1, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    lat_arg = lat_d if num_pages is None else lat_d[:num_pages]
    sm.snapmla_fetch_dequant(lat_arg, sc_d, rope_d, pt_d, cu_d, out)
    torch.cuda.synchronize()
    return out.view(torch.int16).cpu().numpy().view(np.uint16)


def _cache(rng, pages, nan_codes=False):
    lat = rng.integers(0, 256, (pages, 64, 512), dtype=np.uint8)
    if not nan_codes:
        lat[(lat & 0x7F) == 0x7F] = 0x33
    sc = np.exp2(rng.uniform(-40, 12, (pages, 64))).astype(np.float32)
    rope = rng.integers(0, 1 << 16, (pages, 64, 64), dtype=np.uint16)
    return lat, sc, rope


def _cu(lens):
    return np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)


def _assert_equal(got, want, label):
    bad = np.argwhere(got != want)
    assert bad.size == 0, f"{label}: {len(bad)} differing bf16 values, first at row/col {tuple(bad[0])}: " \
        f"got {got[tuple(bad[0])]:#06x} want {want[tuple(bad[0])]:#06x}"


@pytest.mark.parametrize("seed", [0, 1])
def test_ragged_lengths_bitexact(seed):
    rng = np.random.default_rng(100 + seed)
    lens = np.array([0, 1, 63, 64, 65, 200, 129, 4096, 17, 0, 640])
    max_pages = 64
    pages = 300
    lat, sc, rope = _cache(rng, pages)
    pt = np.full((len(lens), max_pages), -7, np.int32)
    perm = rng.permutation(pages)
    k = 0
    for b, n in enumerate(lens):
        npg = (n + 63) // 64
        pt[b, :npg] = perm[k:k + npg]
        k += npg
    cu = _cu(lens)
    print(f"[fetch ragged seed={seed}] rows={cu[-1]} pages used={k}", flush=True)
    _assert_equal(_run(lat, sc, rope, pt, cu), fetch.fetch_dequant(lat, sc, rope, pt, cu), "ragged")


def test_every_code_bitexact():
    # one page holding all 256 codes in every row position, scales spanning the range
    codes = np.tile(np.arange(256, dtype=np.uint8), 2)
    lat = np.stack([np.roll(codes, t) for t in range(64)])[None].astype(np.uint8)
    sc = np.concatenate([[1.0, 2.0 ** -40, 3.0, 0.7], np.exp2(np.linspace(-40, 40, 60))]).astype(np.float32)[None]
    rope = np.arange(64 * 64, dtype=np.uint16).reshape(1, 64, 64)
    pt = np.zeros((1, 1), np.int32)
    cu = _cu([64])
    got = _run(lat, sc, rope, pt, cu)
    _assert_equal(got, fetch.fetch_dequant(lat, sc, rope, pt, cu), "codes")
    assert np.all(got[0, :512][(codes & 0x7F) == 0x7F] == 0x7FC0)      # the two NaN codes


def test_data_errors_nan_rows():
    rng = np.random.default_rng(9)
    pages = 10
    lat, sc, rope = _cache(rng, pages)
    max_pages = 3
    pt = np.array([[0, -1, 2], [pages, 3, 4], [5, 6, 7], [8, 9, 1]], np.int32)
    lens = np.array([150, 130, 200, 64 * 3])     # seq 2 exceeds 3 pages; seq 3 fills them exactly
    cu = _cu(lens)
    got = _run(lat, sc, rope, pt, cu)
    want = fetch.fetch_dequant(lat, sc, rope, pt, cu)
    _assert_equal(got, want, "errors")
    assert np.all(got[cu[2]:cu[3]] == 0x7FC0)
    assert not np.any(got[cu[3]:cu[4], :512] == 0x7FC0)


def test_cache_written_by_append():
    w = wl.custom(B=3, H=16, q_len=1, seq_lens=[700, 64, 1500], seed=23, rotary=True, sigma_tok=1.5)
    from paper_2602_10718_amd.runner import DecodeRunner
    run = DecodeRunner(w, num_splits=8)
    run.append()
    torch.cuda.synchronize()
    cu = _cu(w.seq_lens)
    cu_d = torch.from_numpy(cu.astype(np.int32)).cuda()
    out = torch.empty((int(cu[-1]), 576), dtype=torch.bfloat16, device="cuda")
    sm.snapmla_fetch_dequant(run.kv_latent, run.kv_scale, run.k_rope, run.page_table, cu_d, out)
    torch.cuda.synchronize()
    got = out.view(torch.int16).cpu().numpy().view(np.uint16)
    lat = run.kv_latent.cpu().numpy()
    sc = run.kv_scale.cpu().numpy()
    rope = run.k_rope.view(torch.int16).cpu().numpy().view(np.uint16)
    _assert_equal(got, fetch.fetch_dequant(lat, sc, rope, w.page_table, cu), "append cache")
    # the dequantized latent is the original token within the E4M3 + bf16 roundings
    for b in range(w.B):
        ck, kr = w.tokens(b, 0, int(w.seq_lens[b]))
        x = (ck.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        y = (got[cu[b]:cu[b + 1], :512].astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        sigma = np.max(np.abs(x), axis=1, keepdims=True) / 448
        # E4M3: half an ulp (2^-4 relative; 2^-10 sigma below the normal range), then bf16 (2^-8 relative)
        bound = (2.0 ** -4 + 1.07 * 2.0 ** -8) * np.abs(x) + 1.01 * 2.0 ** -10 * sigma + 1e-30
        assert np.all(np.abs(y - x) <= bound)
        assert np.array_equal(got[cu[b]:cu[b + 1], 512:], kr)


def test_headline_cache_sampled():
    """The bench launch: every sequence of the headline cache, sampled sequences checked bit for bit."""
    w = wl.make("headline")
    from paper_2602_10718_amd.runner import DecodeRunner
    run = DecodeRunner(w)
    cu = _cu(w.seq_lens)
    cu_d = torch.from_numpy(cu.astype(np.int32)).cuda()
    out = torch.empty((int(cu[-1]), 576), dtype=torch.bfloat16, device="cuda")
    print(f"[fetch headline] rows={cu[-1]}", flush=True)
    sm.snapmla_fetch_dequant(run.kv_latent, run.kv_scale, run.k_rope, run.page_table, cu_d, out)
    torch.cuda.synchronize()
    got = out.view(torch.int16)
    for b in (0, w.B // 2, w.B - 1):
        n = int(w.seq_lens[b])
        npg = (n + 63) // 64
        pages = run.page_table[b, :npg].long()
        lat = run.kv_latent[pages].cpu().numpy()
        sc = run.kv_scale[pages].cpu().numpy()
        rope = run.k_rope[pages].view(torch.int16).cpu().numpy().view(np.uint16)
        pt = np.arange(npg, dtype=np.int32)[None]
        want = fetch.fetch_dequant(lat, sc, rope, pt, np.array([0, n]))
        _assert_equal(got[cu[b]:cu[b + 1]].cpu().numpy().view(np.uint16), want, f"headline b={b}")
