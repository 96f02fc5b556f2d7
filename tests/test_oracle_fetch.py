"""Pins of the oracle's fetch-and-dequantize (oracle/fetch.py)."""

import numpy as np
import pytest
import torch

from oracle import e4m3, fetch


def _torch_bf16_bits(x):
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def test_bf16_rounding_matches_torch_cpu():
    rng = np.random.default_rng(7)
    x = (rng.standard_normal(200000) * np.exp2(rng.integers(-60, 60, 200000))).astype(np.float32)
    # values exactly halfway between bf16 neighbours, and just either side of halfway
    base = rng.integers(0x00800000, 0x7F000000, 20000, dtype=np.uint32) & ~np.uint32(0xFFFF)
    half = (base | np.uint32(0x8000)).view(np.float32)
    lo = (base | np.uint32(0x7FFF)).view(np.float32)
    hi = (base | np.uint32(0x8001)).view(np.float32)
    edge = np.array([0.0, -0.0, np.inf, -np.inf, np.finfo(np.float32).max, -np.finfo(np.float32).max,
                     np.finfo(np.float32).tiny, 1e-45, -1e-45, 448.0, -448.0], dtype=np.float32)
    for v in (x, half, -half, lo, hi, edge):
        assert np.array_equal(fetch.f32_to_bf16_bits(v), _torch_bf16_bits(v))


def test_bf16_ties_to_even_by_hand():
    v = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -20, -(1 + 2 ** -8)], dtype=np.float32)
    assert list(fetch.f32_to_bf16_bits(v)) == [0x3F80, 0x3F82, 0x3F81, 0xBF80]
    assert fetch.f32_to_bf16_bits(np.float32(np.nan)) == 0x7FC0


@pytest.mark.parametrize("code,sigma,bits", [
    (0x7E, 1.0, 0x43E0),      # 448
    (0xFE, 1.0, 0xC3E0),      # -448
    (0x7E, 2.0, 0x4460),      # 896
    (0x08, 1.0, 0x3C80),      # 2^-6, smallest normal
    (0x01, 1.0, 0x3B00),      # 2^-9, smallest subnormal
    (0x07, 1.0, 0x3C60),      # 7 * 2^-9 = 0.875 * 2^-6
    (0x80, 1.0, 0x8000),      # -0 stays -0
    (0x00, 3.0, 0x0000),
    (0x38, 2.0 ** -40, 0x2B80),  # 1.0 at the scale floor
])
def test_special_codes(code, sigma, bits):
    codes = np.full((1, 512), code, dtype=np.uint8)
    out = fetch.dequant_rows(codes, np.array([sigma], dtype=np.float32))
    assert np.all(out == bits)


def test_dequant_relative_error_bound():
    rng = np.random.default_rng(3)
    codes = rng.integers(0, 256, (256, 512), dtype=np.uint8)
    codes[(codes & 0x7F) == 0x7F] = 0x11          # no NaN codes in a cache
    sigma = np.exp2(rng.uniform(-30, 10, 256)).astype(np.float32)
    out = fetch.dequant_rows(codes, sigma)
    got = (out.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    exact = e4m3.decode(codes) * sigma.astype(np.float64)[:, None]
    # bf16 keeps 8 significant bits: round-to-nearest error <= 2^-8 relative (plus the float32 step)
    assert np.all(np.abs(got - exact) <= (2.0 ** -8 + 2.0 ** -23) * np.abs(exact))
    assert np.max(np.abs(got - exact) / np.maximum(np.abs(exact), 1e-300)) > 2.0 ** -9   # the bound is reached


def _cache(rng, pages):
    lat = rng.integers(0, 256, (pages, 64, 512), dtype=np.uint8)
    lat[(lat & 0x7F) == 0x7F] = 0x22
    sc = np.exp2(rng.uniform(-8, 4, (pages, 64))).astype(np.float32)
    rope = rng.integers(0, 1 << 16, (pages, 64, 64), dtype=np.uint16)
    return lat, sc, rope


def test_gather_against_per_token_walk():
    rng = np.random.default_rng(11)
    lens = np.array([0, 1, 63, 64, 65, 200, 129])
    max_pages = 4
    pages = 30
    lat, sc, rope = _cache(rng, pages)
    pt = rng.permutation(pages)[:len(lens) * max_pages].reshape(len(lens), max_pages).astype(np.int32)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    out = fetch.fetch_dequant(lat, sc, rope, pt, cu)
    assert out.shape == (lens.sum(), 576)
    for b, n in enumerate(lens):
        for j in range(n):
            page, slot = pt[b, j // 64], j % 64
            row = out[cu[b] + j]
            assert np.array_equal(row[:512], fetch.dequant_rows(lat[page, slot][None], sc[page, slot][None])[0])
            assert np.array_equal(row[512:], rope[page, slot])


def test_data_errors_give_nan_rows():
    rng = np.random.default_rng(5)
    lat, sc, rope = _cache(rng, 8)
    pt = np.array([[0, -1], [8, 1], [2, 3]], dtype=np.int32)      # page -1 and page 8 (== num_pages) are bad
    lens = np.array([100, 70, 129])                                 # the last is longer than 2 pages
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    out = fetch.fetch_dequant(lat, sc, rope, pt, cu)
    assert np.all(out[64:100] == 0x7FC0) and not np.any(out[:64, :512] == 0x7FC0)
    assert np.all(out[100:164] == 0x7FC0) and not np.any(out[164:170, 512:] != rope[1, :6])
    assert np.all(out[170:] == 0x7FC0)
