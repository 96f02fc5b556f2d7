"""Fetch-and-dequantize of the paged FP8 cache into BF16 rows.

Test infrastructure only (see the package docstring).

Definition (Section 3.3, Fused-Fetch-Dequant: for decode phases that reuse
the cache at high precision -- chunk prefill, prefix caching -- the quantized
cache is read and dequantized in one pass).  Sequence b's tokens 0..N_b-1,
N_b = cu[b+1] - cu[b], are written to output rows cu[b] .. cu[b+1]-1, each row
576 bf16 values:

    row[0:512]   = bf16( fp32( D(code_i) * sigma_K ) )    i = 0..511
    row[512:576] = the token's RoPE key, bit for bit

D is the E4M3 decoding (``e4m3.decode``); the product of a 4-significant-bit
value and a float32 scale is exact in float64, so forming it in float64 and
rounding once to float32 equals the float32 product; bf16() rounds to nearest,
ties to even.  Readings (the paper gives the operator's purpose, not its
rounding or layout; these choices are ours): the output keeps the
per-token row layout of the cache (latent then RoPE), the latent is rounded
to bf16 once from the float32 product, NaN becomes the canonical 0x7FC0.
Data errors: a token whose page id lies outside [0, num_pages), and every
token of a sequence longer than max_pages * 64, gets a row of 0x7FC0.

Pinned by tests/test_oracle_fetch.py: bf16 rounding against torch's CPU
conversion and against hand-built ties; special codes (448, the smallest
normal, subnormals, -0) through closed forms; the gather against a per-token
brute-force walk of the page table; the NaN rows of both data errors.
"""

import numpy as np

from . import e4m3

PAGE = 64
D_C = 512
D_R = 64
ROW = D_C + D_R
NAN_BF16 = np.uint16(0x7FC0)


def f32_to_bf16_bits(x):
    """float32 -> bf16 bit patterns, round to nearest, ties to even; NaN -> 0x7FC0."""
    x = np.asarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    r = np.where(np.isnan(x), NAN_BF16, r)
    return r


def dequant_rows(codes, sigma):
    """E4M3 codes [..., 512] and float32 scales [...] -> bf16 bits [..., 512]."""
    v = e4m3.decode(codes) * np.asarray(sigma, dtype=np.float32).astype(np.float64)[..., None]
    with np.errstate(over="ignore", invalid="ignore"):
        return f32_to_bf16_bits(v.astype(np.float32))


def fetch_dequant(kv_latent, kv_scale, k_rope_bits, page_table, cu, num_pages=None):
    """Packed bf16 rows [cu[-1], 576] (uint16 bit patterns) of every sequence's cached tokens.

    kv_latent uint8 [pages, 64, 512], kv_scale float32 [pages, 64], k_rope_bits uint16
    [pages, 64, 64], page_table int32 [B, max_pages], cu int64 [B+1] nondecreasing.
    """
    pages_total = kv_latent.shape[0] if num_pages is None else num_pages
    B, max_pages = page_table.shape
    out = np.empty((int(cu[-1]), ROW), dtype=np.uint16)
    for b in range(B):
        r0, n = int(cu[b]), int(cu[b + 1] - cu[b])
        if n <= 0:
            continue
        if n > max_pages * PAGE:
            out[r0:r0 + n] = NAN_BF16
            continue
        for p in range((n + PAGE - 1) // PAGE):
            t = min(PAGE, n - p * PAGE)
            rows = slice(r0 + p * PAGE, r0 + p * PAGE + t)
            page = int(page_table[b, p])
            if page < 0 or page >= pages_total:
                out[rows] = NAN_BF16
                continue
            out[rows, :D_C] = dequant_rows(kv_latent[page, :t], kv_scale[page, :t])
            out[rows, D_C:] = k_rope_bits[page, :t]
    return out
