"""Seeded synthetic decode workloads shaped like the paper's kernel benchmarks.

This module only draws random inputs: it holds none of the method's
arithmetic (no quantization, no attention) and imports neither the HIP
binding nor the CPU oracle, so both sides can be fed the same bytes.

The paper's kernel studies use batch 32, 16..128 heads, one or two query
tokens per step and KV lengths of 16K..128K (Appendix I; Section 4 efficiency
setup).  Its real KV caches are not available, so values are synthetic: a
content latent concentrated around zero with per-token magnitude spread and a
few outlier channels, and a RoPE key with larger range (the distributions
reported in Section 3.1 motivate these shapes).

Recipe (all values drawn in float32, then rounded to bf16 RNE):
  c_kv[j]   = N(0,1)^512 * lognormal(0, sigma_tok)_j, with 4 seed-chosen
              channels (shared by all tokens of a workload) multiplied by 20
  k_rope[j] = N(0,1)^64, or for "rotary" workloads N(0, var 4)^64 rotated by
              RoPE (base 10000, pairs (i, i+32)) at absolute position j
  q_nope    = N(0,1)^512, q_rope = N(0,1)^64
Random streams are keyed by (seed, sequence, 64-token block) so any token
range of any sequence can be regenerated alone.
"""

from dataclasses import dataclass, field

import numpy as np

PAGE = 64
D_C = 512
D_R = 64


def f32_to_bf16_bits(x):
    """Round float32 values to bf16 (round to nearest even), returning uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (b + np.uint32(0x7FFF) + ((b >> 16) & np.uint32(1))) >> 16
    return r.astype(np.uint16)


def bf16_bits_to_f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass
class Workload:
    name: str
    B: int
    H: int
    q_len: int
    causal: bool
    seq_lens: np.ndarray            # int32 [B]: cached tokens incl. the current step's tokens
    n_new: int                      # tokens appended per sequence per step
    sigma_tok: float                # lognormal sigma of the per-token latent magnitude
    rotary: bool                    # k_rope = RoPE(N(0, var 4)) by absolute position
    seed: int
    tau: float = 1.0 / np.sqrt(192.0)
    kv_chunk_tokens: int = 0        # 0: balanced split plan; >0: fixed chunks per sequence
    shuffle_pages: bool = True
    page_table: np.ndarray = field(default=None, repr=False)
    num_pages: int = 0
    outliers: np.ndarray = field(default=None, repr=False)
    content_scale: float = 1.0      # multiplies every content value
    rope_scale: float = 1.0         # multiplies every RoPE key value
    q_rope_scale: float = 1.0       # multiplies every q_rope value
    q_nope_scale: float = 1.0       # multiplies every q_nope value
    outlier_gain: float = 20.0      # gain of the 4 outlier content channels

    @property
    def rows(self):
        return self.H * self.q_len

    @property
    def max_pages(self):
        return self.page_table.shape[1]

    @property
    def total_tokens(self):
        return int(np.sum(self.seq_lens))

    def kv_bytes(self):
        """Bytes of cache read by one decode step: 512 B latent + 128 B rope + 4 B scale per token."""
        return self.total_tokens * (D_C + 2 * D_R + 4)

    # ---- per-token content -------------------------------------------------
    def tokens(self, b, t0, t1):
        """bf16 bits of c_kv [t1-t0, 512] and k_rope [t1-t0, 64] for tokens t0..t1-1 of sequence b."""
        ck = np.empty((t1 - t0, D_C), np.uint16)
        kr = np.empty((t1 - t0, D_R), np.uint16)
        k0 = t0 // PAGE
        k1 = (t1 + PAGE - 1) // PAGE
        for k in range(k0, k1):
            c, r = self._block(b, k)
            a = max(t0, k * PAGE)
            z = min(t1, (k + 1) * PAGE)
            ck[a - t0:z - t0] = c[a - k * PAGE:z - k * PAGE]
            kr[a - t0:z - t0] = r[a - k * PAGE:z - k * PAGE]
        return ck, kr

    def _block(self, b, k):
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([self.seed, 1, b, k])))
        z = rng.standard_normal((PAGE, D_C), dtype=np.float32)
        lam = np.exp(rng.standard_normal(PAGE, dtype=np.float32) * np.float32(self.sigma_tok))
        z *= lam[:, None]
        z[:, self.outliers] *= np.float32(self.outlier_gain)
        if self.content_scale != 1.0:
            z *= np.float32(self.content_scale)
        if self.rotary:
            x = rng.standard_normal((PAGE, D_R), dtype=np.float32) * np.float32(2.0)
            pos = (k * PAGE + np.arange(PAGE)).astype(np.float64)
            theta = 10000.0 ** (-np.arange(D_R // 2) / (D_R // 2))
            ang = pos[:, None] * theta[None, :]
            c, s = np.cos(ang), np.sin(ang)
            x1, x2 = x[:, : D_R // 2].astype(np.float64), x[:, D_R // 2:].astype(np.float64)
            r = np.concatenate([x1 * c - x2 * s, x1 * s + x2 * c], axis=1).astype(np.float32)
        else:
            r = rng.standard_normal((PAGE, D_R), dtype=np.float32)
        if self.rope_scale != 1.0:
            r = r * np.float32(self.rope_scale)
        return f32_to_bf16_bits(z), f32_to_bf16_bits(r)

    # ---- queries -----------------------------------------------------------
    def queries(self):
        """bf16 bits of q_nope [B, q_len, H, 512] and q_rope [B, q_len, H, 64]."""
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([self.seed, 2])))
        qn = rng.standard_normal((self.B, self.q_len, self.H, D_C), dtype=np.float32)
        if self.q_nope_scale != 1.0:
            qn = qn * np.float32(self.q_nope_scale)
        qr = rng.standard_normal((self.B, self.q_len, self.H, D_R), dtype=np.float32)
        if self.q_rope_scale != 1.0:
            qr = qr * np.float32(self.q_rope_scale)
        return f32_to_bf16_bits(qn), f32_to_bf16_bits(qr)


def _finish(w):
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.seed, 3])))
    w.outliers = np.sort(rng.choice(D_C, size=4, replace=False))
    npg = (w.seq_lens + PAGE - 1) // PAGE
    total = int(np.sum(npg))
    maxp = max(1, int(np.max(npg)) if len(npg) else 1)
    phys = rng.permutation(total) if w.shuffle_pages else np.arange(total)
    pt = np.full((w.B, maxp), -1, np.int32)
    o = 0
    for b in range(w.B):
        pt[b, : npg[b]] = phys[o:o + npg[b]]
        o += npg[b]
    w.page_table = pt
    w.num_pages = max(total, 1)
    return w


# The five workloads, by name: what each is, and the seed its inputs come from.
WORKLOADS = {
    "tiny": ("tiny B1 H16 ctx256", 1001),
    "dsv3": ("dsv3-shaped B32 H128 ctx4096", 1002),
    "headline": ("64-head ragged 8K-32K B64", 1003),
    "longsplit": ("long split B8 H64 ctx128K x32 chunks", 1004),
    "mtp": ("MTP B128 H128 q_len2 causal ragged 1K-16K", 1005),
}


def describe(name):
    """One-line description of workload `name`."""
    return WORKLOADS[name][0]


def make(name, seed=None, B=None, ctx=None, ctx_range=None):
    """Build workload `name` (a key of WORKLOADS).  B / ctx / ctx_range shrink it for fast tests."""
    if name not in WORKLOADS:
        raise ValueError(f"unknown workload {name!r}; one of {sorted(WORKLOADS)}")
    seed = WORKLOADS[name][1] if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0])))
    if name == "tiny":
        b = B or 1
        w = Workload("tiny", b, 16, 1, False, np.full(b, ctx or 256, np.int32), 1, 1.0, False, seed,
                     shuffle_pages=False)
    elif name == "dsv3":
        b = B or 32
        w = Workload("dsv3", b, 128, 1, False, np.full(b, ctx or 4096, np.int32), 1, 1.0, False, seed)
    elif name == "headline":
        b = B or 64
        lo, hi = ctx_range or (8192, 32768)
        w = Workload("headline", b, 64, 1, False, rng.integers(lo, hi + 1, b).astype(np.int32), 1, 1.5,
                     True, seed)
    elif name == "longsplit":
        b = B or 8
        w = Workload("longsplit", b, 64, 1, False, np.full(b, ctx or 131072, np.int32), 1, 1.0, False, seed,
                     kv_chunk_tokens=4096)
    else:   # "mtp"
        b = B or 128
        lo, hi = ctx_range or (1024, 16384)
        w = Workload("mtp", b, 128, 2, True, rng.integers(lo, hi + 1, b).astype(np.int32), 2, 1.0, False,
                     seed)
    return _finish(w)


def custom(B, H, q_len, seq_lens, causal=False, sigma_tok=1.0, rotary=False, seed=7, n_new=1,
           shuffle_pages=True, kv_chunk_tokens=0):
    """A workload with explicit shapes (edge cases: ragged tails, empty sequences, ...)."""
    w = Workload("custom", B, H, q_len, causal, np.asarray(seq_lens, np.int32), n_new, sigma_tok, rotary,
                 seed, kv_chunk_tokens=kv_chunk_tokens, shuffle_pages=shuffle_pages)
    return _finish(w)


SWEEP_HEADS = (16, 32, 64, 128)
SWEEP_QLEN = (1, 2)


def sweep(H, q_len, seed=1100, B=32, ctx_range=(16384, 131072)):
    """The sensitivity-sweep workload: batch 32, lengths U[16K, 128K], H heads, q_len query tokens
    (causal when q_len == 2).  The cache content and page table depend only on the seed, B and the
    lengths, so every (H, q_len) of the sweep reads the same cache."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0])))
    lens = rng.integers(ctx_range[0], ctx_range[1] + 1, B).astype(np.int32)
    w = Workload("sweep", B, H, q_len, q_len == 2, lens, q_len, 1.5, True, seed)
    return _finish(w)


def ablation(B=8, H=16, ctx=4096, seed=1200):
    """The quantization-granularity ablation workload: content around 10^0-10^1 with per-token
    lognormal(0, 1) magnitudes and 4 outlier channels x20, RoPE keys around 10^3 (a rotary
    rotation of N(0, var 4) vectors scaled by 250) -- the magnitude relation the paper reports for
    real caches (content ~10^1, RoPE ~10^3).  Queries: q_nope x 0.1, q_rope x 1/50, so that the
    logits spread over a few units and the RoPE term carries about as much as the content term."""
    w = Workload("ablation", B, H, 1, False, np.full(B, ctx, np.int32), 1, 1.0, True, seed,
                 content_scale=3.0, rope_scale=250.0, q_rope_scale=1.0 / 50.0, q_nope_scale=0.1)
    return _finish(w)
