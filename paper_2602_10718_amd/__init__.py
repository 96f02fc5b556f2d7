"""SnapMLA FP8 MLA decode for MI355X (gfx950).

The compute path is the HIP library ``libsnapmla.so`` (sources in ``csrc/``,
C declarations in ``include/snapmla.h``).  ``paper_2602_10718_amd.snapmla``
is the thin ctypes binding with the same function names; ``workloads``
draws the seeded synthetic inputs.  Importing this package loads nothing;
importing ``snapmla`` loads the library and fails loudly if it is missing.
"""
