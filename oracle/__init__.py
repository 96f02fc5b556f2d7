"""CPU oracle for the SnapMLA FP8 MLA decode path -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, float64 numpy statement of what the decode
path computes.  It exists so that tests, the smoke check and the benchmark's
CPU-baseline leg can check the HIP library against an independent
definition.  Nothing on the product path may import it; it shares no code,
tables or constants with the HIP library (``paper_2602_10718_amd``), and it
never imports that package.

Modules
-------
e4m3     OCP E4M3 (``FN`` variant, max 448) codec written from the format
         definition, plus brute-force helpers used to pin it.
quant    the per-token row quantizer (Appendix C, per-token equation; the
         scale rule the paper uses for P in Algorithm 1).
fetch    fetch-and-dequantize of the paged cache into BF16 rows (Section 3.3,
         Fused-Fetch-Dequant).
granularity  the KV-cache quantization granularities of the accuracy ablation
         (Appendix G, Table 3) and its three error metrics.
mla      absorbed-mode MLA decode over per-token FP8 content + BF16 RoPE
         (Section 2 absorbed score; Section 3.2; Appendix D recurrences;
         Algorithm 1 finalisation), the split-KV log-sum-exp merge, and the
         unquantized BF16 reference.

Parity status of each function is stated in its docstring; anything not
pinned by an independent check says "parity unpinned".
"""

from . import e4m3, quant, mla, fetch, granularity  # noqa: F401

EPS = quant.EPS
