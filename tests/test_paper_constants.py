"""The oracle's constants against the values the paper prints (tests/golden/paper_constants.txt)."""

import os

from oracle import e4m3, mla

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_constants.txt")


def _load():
    out = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        name, val = line.split()[:2]
        out[name] = float(val)
    return out


def test_constants_match_paper():
    g = _load()
    assert mla.FP8_MAX == g["fp8_max"] == e4m3.MAX
    assert mla.BLOCK == g["block_n"]
    assert e4m3.decode_table()[0x7E] == g["fp8_max"]
    # the effective-peak derivation of the roofline appendix
    assert round(g["bf16_peak_tflops"] * (16 + 1) / (16 / 2 + 1), 1) == g["effective_peak_tflops"]
    assert g["d_c"] == 8 * 64 and g["d_r"] == 64
