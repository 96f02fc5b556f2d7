"""Host-side checks of the seeded workload generator (no method arithmetic here)."""

import numpy as np

from paper_2602_10718_amd import workloads as wl


def test_configs_shapes_and_page_tables():
    for name in wl.WORKLOADS:
        w = wl.make(name)
        assert w.seq_lens.shape == (w.B,)
        npg = (w.seq_lens + 63) // 64
        pt = w.page_table
        used = np.concatenate([pt[b, :npg[b]] for b in range(w.B)])
        assert np.array_equal(np.sort(used), np.arange(w.num_pages))   # every physical page once
        assert np.all(pt[np.arange(pt.shape[1])[None, :] >= npg[:, None]] == -1)
    w3 = wl.make("headline")
    assert w3.seq_lens.min() >= 8192 and w3.seq_lens.max() <= 32768 and w3.H == 64
    w5 = wl.make("mtp")
    assert w5.q_len == 2 and w5.causal and w5.rows == 256


def test_token_ranges_regenerate_identically():
    w = wl.make("headline", B=2, ctx_range=(300, 400))
    a, ra = w.tokens(1, 0, 300)
    b, rb = w.tokens(1, 100, 230)
    assert np.array_equal(a[100:230], b) and np.array_equal(ra[100:230], rb)
    w2 = wl.make("headline", B=2, ctx_range=(300, 400))
    assert np.array_equal(w2.tokens(1, 0, 300)[0], a)
    q1 = w.queries()
    assert q1[0].shape == (2, 1, 64, 512) and q1[1].shape == (2, 1, 64, 64)


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1e-30], np.float32)
    b = wl.f32_to_bf16_bits(x)
    y = wl.bf16_bits_to_f32(b)
    assert y[0] == 1.0 and y[1] == 1.0 and y[2] == 1.0 + 2 ** -6 and y[3] == -2.5
    rng = np.random.default_rng(0)
    z = rng.standard_normal(10000).astype(np.float32)
    bz = wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(z))
    assert np.all(np.abs(bz - z) <= np.abs(z) * 2 ** -8)
