"""Per-token (per-row) FP8 quantizer of the content latent and of q_nope.

Test infrastructure only (see the package docstring).

Definition (Appendix C, per-token quantization: one scale per row,
X_q = round(X / S); Section 3.1, per-token granularity for the content part
only; Appendix D: dynamic scales are floored by a small epsilon before
division).  For one row x of bf16 values:

    a     = max_i |x_i|                         (exact)
    sigma = max( fp32(a / 448), EPS )           (IEEE float32 division, RNE)
    y_i   = fp32(x_i / sigma)                   (IEEE float32 division, RNE)
    code_i = E4M3(y_i)                          (RNE, satfinite)

Readings (the paper does not fix these; these choices are ours):
  * the per-token scale is amax/448, the same rule Algorithm 1 uses for the
    probability blocks;
  * the quotient is formed in float32 and then rounded to E4M3 -- two
    roundings, deliberately;
  * EPS = 2^-40.

Pinned by tests/test_oracle_quant.py: the amax element maps to +-448, the
reconstruction error obeys the E4M3 half-ulp bound, scaling a row by 2^k
scales sigma by 2^k and keeps the codes, an all-zero row gives sigma = EPS and
zero codes.
"""

import numpy as np

from . import e4m3

EPS = np.float32(2.0 ** -40)
_F448 = np.float32(448.0)


def bf16_to_f32(bits):
    """bf16 bit patterns (uint16) -> float32, exact."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32)


def quantize_rows(x_bits):
    """Quantize rows of bf16 bit patterns.

    Parameters
    ----------
    x_bits : uint16 array [..., n]  bf16 bit patterns, one row per token/query row.

    Returns
    -------
    codes : uint8 [..., n]   E4M3 codes
    sigma : float32 [...]    per-row scale; the row is reconstructed as sigma * decode(codes)
    """
    x = bf16_to_f32(x_bits)
    a = np.max(np.abs(x), axis=-1)
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        sigma = np.maximum(a / _F448, EPS).astype(np.float32)
        y = (x / sigma[..., None]).astype(np.float32)
    codes = e4m3.encode(y)
    return codes, sigma
