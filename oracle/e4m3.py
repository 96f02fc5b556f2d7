"""OCP FP8 E4M3 codec (the "FN" variant with max 448), float64, from the format definition.

Test infrastructure only (see the package docstring).

Format (OCP 8-bit floating point specification, E4M3): 1 sign bit, 4 exponent
bits with bias 7, 3 mantissa bits.  Exponent field 0 encodes subnormals
m/8 * 2^-6; exponent fields 1..15 encode (1 + m/8) * 2^(E-7), except that
exponent 15 with mantissa 7 (codes 0x7F / 0xFF) is NaN.  There is no infinity;
the largest finite magnitude is 448 (code 0x7E).  The paper quantizes the
content cache and the fused probability blocks to this format (Section 4
setup names E4M3; Algorithm 1 divides block maxima by 448).

Encoding is round-to-nearest, ties to the even mantissa, with saturation of
finite overflow to +-448 ("satfinite"); the sign of zero is kept
(-0.0 -> 0x80); NaN maps to 0x7F.

Pinned by tests/test_oracle_e4m3.py against (a) values fixed by the format
definition and (b) a brute-force nearest-value search over the 254 finite
codes.
"""

import numpy as np

MAX = 448.0
# the smallest magnitude of the normal range and the subnormal quantum
MIN_NORMAL = 2.0 ** -6
SUB_QUANTUM = 2.0 ** -9


def _decode_one(c):
    sign = -1.0 if c & 0x80 else 1.0
    e = (c >> 3) & 0xF
    m = c & 0x7
    if e == 0xF and m == 0x7:
        return np.nan
    if e == 0:
        return sign * (m / 8.0) * 2.0 ** -6
    return sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)


_TABLE = np.array([_decode_one(c) for c in range(256)], dtype=np.float64)


def decode_table():
    """float64[256]: the value of every code (NaN for 0x7F and 0xFF)."""
    return _TABLE.copy()


def decode(codes):
    """Decode uint8 codes to float64 values (exact)."""
    return _TABLE[np.asarray(codes, dtype=np.uint8)]


def encode(x):
    """Round float64 (or float32) values to E4M3 codes: RNE, satfinite, signed zero.

    The input is taken at its exact value (float32 inputs are widened without
    rounding), so a float32 quotient is rounded exactly once here.
    """
    x = np.asarray(x, dtype=np.float64)
    shape = x.shape
    x = x.reshape(-1)
    out = np.zeros(x.shape, dtype=np.uint8)
    nan = np.isnan(x)
    sign = np.signbit(x) & ~nan
    a = np.abs(np.where(nan, 0.0, x))
    # exponent of the quantum: normal binade e has quantum 2^(e-3); below 2^-6
    # the quantum is fixed at 2^-9
    safe = np.where(a > 0, a, 1.0)
    _, fexp = np.frexp(safe)            # safe = f * 2^fexp, f in [0.5, 1)
    e = np.maximum(fexp - 1, -6)        # floor(log2 a), clamped to the subnormal binade
    quantum = np.ldexp(1.0, e - 3)
    n = np.rint(a / quantum)            # a / quantum is exact; rint is ties-to-even
    v = n * quantum                     # rounded magnitude (exact)
    v = np.where(a >= 464.0, MAX, np.minimum(v, MAX))   # satfinite (464 ties to 448, even)
    # re-encode the rounded magnitude exactly
    code = np.zeros(x.shape, dtype=np.int64)
    sub = v < MIN_NORMAL
    code[sub] = np.rint(v[sub] / SUB_QUANTUM).astype(np.int64)
    vn = np.where(sub, 1.0, v)
    _, ve = np.frexp(vn)
    E = ve - 1                          # v = (1 + m/8) * 2^E
    mant = np.rint((vn / np.ldexp(1.0, E) - 1.0) * 8.0).astype(np.int64)
    code[~sub] = ((E[~sub] + 7) << 3) | mant[~sub]
    out[:] = code.astype(np.uint8)
    out[sign] |= 0x80
    out[nan] = 0x7F
    return out.reshape(shape)


def finite_values():
    """The sorted distinct non-negative finite values (0 and the 126 positive ones)."""
    t = _TABLE[:0x7F]
    return np.unique(t[~np.isnan(t)])


def encode_bruteforce(x):
    """Reference encoder by exhaustive search (slow; for pinning ``encode``).

    For each input, pick among all finite codes the one whose value is nearest;
    on an exact tie pick the code with an even mantissa (lowest bit 0);
    magnitudes at or beyond the 448/480 midpoint saturate to 448.
    """
    x = np.asarray(x, dtype=np.float64).reshape(-1)
    codes = np.array([c for c in range(256) if not np.isnan(_TABLE[c])], dtype=np.int64)
    vals = _TABLE[codes]
    out = np.zeros(x.shape, dtype=np.uint8)
    for i, xi in enumerate(x):
        if np.isnan(xi):
            out[i] = 0x7F
            continue
        neg = np.signbit(xi)
        a = abs(xi)
        if a >= 464.0:
            out[i] = 0x7E | (0x80 if neg else 0)
            continue
        pos = codes[(vals >= 0) & ~np.signbit(vals)]
        pv = _TABLE[pos]
        d = np.abs(pv - a)
        best = np.flatnonzero(d == d.min())
        if len(best) > 1:
            even = [b for b in best if (pos[b] & 1) == 0]
            best = even
        c = int(pos[best[0]])
        out[i] = c | (0x80 if neg else 0)
    return out


def fp32_thresholds():
    """For each positive code k = 1..126 the smallest float32 value that encodes to k.

    Returned as uint32 bit patterns (ascending).  A non-negative float32 x below
    464 encodes to the number of thresholds <= bits(x), which allows checking an
    encoder against this codec over every float32 pattern without evaluating the
    codec per pattern.
    """
    vals = finite_values()              # 0, 2^-9, ..., 448
    th = np.zeros(len(vals) - 1, dtype=np.uint32)
    for k in range(1, len(vals)):
        mid = np.float32((vals[k - 1] + vals[k]) / 2.0)   # exact: at most 5 significant bits
        assert float(mid) == (vals[k - 1] + vals[k]) / 2.0
        code_at_mid = int(encode(np.float64(mid)))
        bits = np.array([mid], dtype=np.float32).view(np.uint32)[0]
        th[k - 1] = bits if code_at_mid == k else bits + 1
    return th
