"""KV-cache quantization granularities of the numerical-accuracy ablation (Appendix G, Table 3).

Test infrastructure only (see the package docstring).

Every configuration turns the bf16 cache rows of a batch -- content c [N, 512],
RoPE key r [N, 64] per sequence -- into the planes the decode path reads: E4M3
codes, one float32 scale per token (the content row is sigma_j * D(code_j)) and a
bf16 RoPE row.  Scales are max(fp32(amax / 448), EPS) over the configuration's
group and every quotient is an IEEE float32 division rounded to E4M3, as in the
per-token quantizer (``quant.quantize_rows``):

    snapmla  per-token content, RoPE kept in bf16               (the method)
    A        per-token over the whole 576-d row, RoPE quantized too (RoPE-unaware)
    B        per-tensor static: scale 1.0, RoPE in bf16
    C        per-tensor dynamic: one scale over every content value of the batch
    D        per-block: one scale per 64-token block (page) of a sequence

Readings (the table names the granularities only; these choices are ours):
the "tensor" of C is the cache of the whole batch; the blocks of D are the
64-token pages, aligned to position 0; in A the RoPE part shares the token's
scale and the decode path reads it back as bf16(fp32(sigma * D(code))).

``scores`` gives the three metrics of the ablation for an output against the
bf16 reference: RMSE over all elements, the mean over rows of 1 - cosine
similarity, and the relative L2 error of the whole output.

Pinned by tests/test_oracle_granularity.py: "snapmla" equals the per-token
quantizer; each configuration's scales by closed form on constructed rows (a
row with the batch maximum, a block maximum, scale 1.0 saturating at 448); A's
RoPE reconstruction within the E4M3 half-ulp; the metrics on hand-computed
vectors.
"""

import numpy as np

from . import e4m3, quant
from .fetch import f32_to_bf16_bits

CONFIGS = ("snapmla", "A", "B", "C", "D")
PAGE = 64
_F448 = np.float32(448.0)


def _bf16_to_f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _scale(amax):
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        return np.maximum(np.asarray(amax, dtype=np.float32) / _F448, quant.EPS).astype(np.float32)


def _codes(x, sigma):
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        return e4m3.encode((x / sigma[..., None]).astype(np.float32))


def quantize(config, seqs):
    """seqs: list of (c_bits uint16 [N, 512], r_bits uint16 [N, 64]) per sequence.

    Returns a list of (codes uint8 [N, 512], sigma float32 [N], rope_bits uint16 [N, 64]).
    """
    if config not in CONFIGS:
        raise ValueError(config)
    out = []
    if config == "C":
        amax_all = max((float(np.max(np.abs(_bf16_to_f32(c)))) if len(c) else 0.0) for c, _ in seqs)
        sig_all = _scale(np.float32(amax_all))
    for c_bits, r_bits in seqs:
        c = _bf16_to_f32(c_bits)
        n = c.shape[0]
        r_out = np.array(r_bits, dtype=np.uint16, copy=True)
        if config == "snapmla":
            codes, sigma = quant.quantize_rows(c_bits)
        elif config == "A":
            r = _bf16_to_f32(r_bits)
            sigma = _scale(np.maximum(np.max(np.abs(c), axis=1), np.max(np.abs(r), axis=1)))
            codes = _codes(c, sigma)
            rq = e4m3.decode(_codes(r, sigma)) * sigma.astype(np.float64)[:, None]
            r_out = f32_to_bf16_bits(rq.astype(np.float32))
        elif config == "B":
            sigma = np.ones(n, dtype=np.float32)
            codes = _codes(c, sigma)
        elif config == "C":
            sigma = np.full(n, sig_all, dtype=np.float32)
            codes = _codes(c, sigma)
        else:  # "D"
            sigma = np.empty(n, dtype=np.float32)
            for k in range(0, n, PAGE):
                sigma[k:k + PAGE] = _scale(np.max(np.abs(c[k:k + PAGE])))
            codes = _codes(c, sigma)
        out.append((codes, sigma, r_out))
    return out


def scores(o, ref):
    """RMSE, mean over rows of (1 - cosine similarity), relative L2 of o against ref ([rows, d])."""
    o = np.asarray(o, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    d = o - ref
    rmse = float(np.sqrt(np.mean(d * d)))
    num = np.sum(o * ref, axis=1)
    den = np.linalg.norm(o, axis=1) * np.linalg.norm(ref, axis=1)
    ok = den > 0
    cosd = float(np.mean(1.0 - num[ok] / den[ok])) if np.any(ok) else 0.0
    rel = float(np.linalg.norm(d) / max(np.linalg.norm(ref), 1e-300))
    return {"rmse": rmse, "cos_diff": cosd, "rel_l2": rel}
