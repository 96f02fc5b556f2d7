"""Pins of the oracle's per-token quantizer by invariants of the definition."""

import numpy as np

from paper_2602_10718_amd import workloads as wl
from oracle import e4m3, quant
from paper_2602_10718_amd.workloads import f32_to_bf16_bits, bf16_bits_to_f32


def _rows(rng, n=64, d=512, spread=True):
    x = rng.standard_normal((n, d)).astype(np.float32)
    if spread:
        x *= np.exp(rng.standard_normal(n) * 1.5).astype(np.float32)[:, None]
        x[:, [3, 100, 257, 511]] *= 20
    return f32_to_bf16_bits(x)


def test_amax_maps_to_448_and_sign():
    rng = np.random.default_rng(1)
    bits = _rows(rng)
    codes, sigma = quant.quantize_rows(bits)
    x = bf16_bits_to_f32(bits)
    am = np.argmax(np.abs(x), axis=1)
    top = codes[np.arange(len(am)), am]
    assert np.all((top & 0x7F) == 0x7E)
    assert np.array_equal(top >> 7, (x[np.arange(len(am)), am] < 0).astype(np.uint8))
    assert sigma.dtype == np.float32


def test_reconstruction_error_bound():
    rng = np.random.default_rng(2)
    bits = _rows(rng, n=128)
    codes, sigma = quant.quantize_rows(bits)
    x = bf16_bits_to_f32(bits).astype(np.float64)
    xh = e4m3.decode(codes) * sigma.astype(np.float64)[:, None]
    y = np.abs(x) / sigma.astype(np.float64)[:, None]
    err = np.abs(xh - x)
    normal = y >= 2.0 ** -6
    # E4M3 half-ulp bound (2^-4 relative in the normal range, 2^-10 absolute in
    # units of sigma below it) plus the float32 rounding of the quotient
    assert np.all(err[normal] <= (2.0 ** -4 + 2.0 ** -22) * np.abs(x[normal]))
    sub_bound = (2.0 ** -10 + 2.0 ** -22) * np.broadcast_to(sigma.astype(np.float64)[:, None], x.shape)
    assert np.all(err[~normal] <= sub_bound[~normal])


def test_power_of_two_scaling_is_exact():
    rng = np.random.default_rng(3)
    bits = _rows(rng, n=32, spread=False)
    codes, sigma = quant.quantize_rows(bits)
    x = bf16_bits_to_f32(bits)
    for k in (-5, -1, 1, 7):
        xs = f32_to_bf16_bits(x * np.float32(2.0 ** k))      # exact: power-of-two scaling of bf16
        c2, s2 = quant.quantize_rows(xs)
        assert np.array_equal(c2, codes)
        assert np.array_equal(s2, (sigma * np.float32(2.0 ** k)).astype(np.float32))


def test_zero_row_and_tiny_row():
    bits = np.zeros((2, 512), np.uint16)
    bits[1, 7] = f32_to_bf16_bits(np.array([1e-20], np.float32))[0]
    codes, sigma = quant.quantize_rows(bits)
    assert sigma[0] == quant.EPS and np.all(codes[0] == 0)
    # below the floor the scale stays EPS; 1e-20 / 2^-40 is far below the smallest
    # E4M3 subnormal, so the code is zero
    assert sigma[1] == quant.EPS
    assert np.all(codes[1] == 0)
    # a value just above the floor keeps its magnitude on the E4M3 grid in units of EPS
    bits = np.zeros((1, 512), np.uint16)
    bits[0, 0] = f32_to_bf16_bits(np.array([300 * 2.0 ** -40], np.float32))[0]
    c, s = quant.quantize_rows(bits)
    assert s[0] == quant.EPS and e4m3.decode(c[0, 0]) == 288.0   # 300 rounds to 288 on the grid


def test_two_roundings_reading():
    """The quantizer rounds the float32 quotient x / sigma to E4M3 (two roundings), not the exact
    quotient.  A constructed bf16 row where the readings differ: amax 260 gives sigma =
    fp32(260 / 448) = 0.58035713..., slightly below 65/112, so 195 / sigma lies just above 336 --
    the midpoint between the E4M3 values 320 (mantissa 2, even) and 352.  In float32 the quotient
    rounds to exactly 336, a tie that goes to 320; rounded once it would give 352."""
    row = np.zeros(512, np.float32)
    row[0], row[1] = 260.0, 195.0
    codes, sigma = quant.quantize_rows(wl.f32_to_bf16_bits(row)[None])
    assert sigma[0] == np.float32(260.0) / np.float32(448.0)
    assert np.float32(np.float32(195.0) / sigma[0]) == np.float32(336.0)      # the float32 quotient: a tie
    assert 195.0 / float(sigma[0]) > 336.0                                     # the exact one: above it
    assert codes[0, 0] == 0x7E                                                  # 448
    assert e4m3.decode(codes[0, 1:2])[0] == 320.0
    assert codes[0, 1] == 0x7A                                                  # 0 1111 010: 1.25 * 2^8


def test_metrics_closed_forms():
    from oracle import check
    rng = np.random.default_rng(5)
    o = rng.standard_normal((6, 512))
    lse = rng.standard_normal(6) * 10
    m = check.metrics(o * 1.01, lse + 0.25, o, lse)
    assert abs(m["rel_l2"] - 0.01) < 1e-12
    assert abs(m["one_minus_cos"]) < 1e-12
    assert abs(m["lse_max_abs"] - 0.25) < 1e-12
    assert abs(m["max_abs"] - 0.01 * np.max(np.abs(o))) < 1e-12
    assert abs(m["rmse"] - 0.01 * np.sqrt(np.mean(o ** 2))) < 1e-12
    # an orthogonal error of equal norm: 1 - cos = 1 - 1/sqrt(2) in that row
    v = np.zeros((1, 4))
    v[0, 0] = 1.0
    w = np.zeros((1, 4))
    w[0, :2] = 1.0
    m2 = check.metrics(w, np.zeros(1), v, np.zeros(1))
    assert abs(m2["one_minus_cos"] - (1 - 1 / np.sqrt(2))) < 1e-12
