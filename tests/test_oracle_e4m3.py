"""Pins of the oracle's E4M3 codec against the format definition and brute force."""

import numpy as np

from oracle import e4m3


def test_decode_table_matches_format_definition():
    t = e4m3.decode_table()
    # values the OCP E4M3 definition fixes
    assert t[0x00] == 0.0 and np.signbit(t[0x80])
    assert t[0x01] == 2.0 ** -9            # smallest subnormal
    assert t[0x07] == 7.0 / 8 * 2.0 ** -6  # largest subnormal
    assert t[0x08] == 2.0 ** -6            # smallest normal
    assert t[0x38] == 1.0
    assert t[0x7E] == 448.0 and t[0xFE] == -448.0
    assert np.isnan(t[0x7F]) and np.isnan(t[0xFF])
    assert t[0x77] == 240.0                # exponent field 14, mantissa 7: 1.875 * 2^7
    assert t[0x78] == 256.0                # exponent field 15 is an ordinary binade in E4M3
    finite = t[~np.isnan(t)]
    assert len(finite) == 254
    pos = t[:0x7F]
    assert np.all(np.diff(pos) > 0)        # codes 0x00..0x7E increase strictly
    assert np.array_equal(t[0x80:0xFF], -t[0x00:0x7F])


def _grid_and_midpoints():
    v = e4m3.finite_values()
    mids = (v[:-1] + v[1:]) / 2
    return v, mids


def test_encode_matches_bruteforce():
    v, mids = _grid_and_midpoints()
    rng = np.random.default_rng(0)
    xs = np.concatenate([
        v, -v, mids, -mids,
        mids * (1 + 2.0 ** -20), mids * (1 - 2.0 ** -20),
        -mids * (1 + 2.0 ** -20),
        rng.uniform(-460, 460, 3000),
        rng.standard_normal(2000) * np.exp(rng.uniform(-14, 6, 2000)),
        [448.0, 460.0, 463.999, 464.0, 470.0, 1e9, -1e9, 0.0, -0.0, 2.0 ** -10, 2.0 ** -11, 1e-30],
    ])
    assert np.array_equal(e4m3.encode(xs), e4m3.encode_bruteforce(xs))


def test_encode_ties_go_to_even_mantissa():
    v, mids = _grid_and_midpoints()
    codes = e4m3.encode(mids)
    assert np.all(codes & 1 == 0)
    assert e4m3.encode(2.0 ** -10) == 0x00              # tie between 0 and 2^-9
    assert e4m3.encode(3 * 2.0 ** -10) == 0x02          # tie between 2^-9 (odd) and 2^-8 (even)
    assert e4m3.encode(15.0 / 16 * 2.0 ** -6) == 0x08   # largest subnormal / smallest normal tie


def test_encode_special_values():
    assert e4m3.encode(-0.0) == 0x80
    assert e4m3.encode(np.nan) == 0x7F
    assert e4m3.encode(464.0) == 0x7E and e4m3.encode(1e30) == 0x7E and e4m3.encode(-1e30) == 0xFE
    assert e4m3.encode(-1e-30) == 0x80
    x = np.array([[1.0, -2.0], [0.5, 448.0]])
    assert e4m3.encode(x).shape == (2, 2)


def test_roundtrip_of_every_finite_code():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
    assert np.array_equal(e4m3.encode(e4m3.decode(codes)), codes)


def test_fp32_thresholds():
    th = e4m3.fp32_thresholds()
    assert len(th) == 126 and np.all(np.diff(th.astype(np.int64)) > 0)
    f = th.view(np.float32).astype(np.float64)
    below = (th - 1).view(np.float32).astype(np.float64)
    k = np.arange(1, 127)
    assert np.array_equal(e4m3.encode(f).astype(np.int64), k)
    assert np.array_equal(e4m3.encode(below).astype(np.int64), k - 1)


def test_dense_float32_sweep_against_thresholds():
    # every 37th float32 pattern below 464 (about 30M values) in 8 slices
    th = e4m3.fp32_thresholds().astype(np.int64)
    top = int(np.array([464.0], np.float32).view(np.uint32)[0])
    for s in range(8):
        pats = np.arange(s, top, 37 * 8, dtype=np.int64)
        x = pats.astype(np.uint32).view(np.float32).astype(np.float64)
        expect = np.searchsorted(th, pats, side="right")
        assert np.array_equal(e4m3.encode(x).astype(np.int64), expect)
