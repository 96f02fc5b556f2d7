"""Host-only checks of the C ABI: the library loads, exports what include/snapmla.h declares,
and rejects bad arguments with the documented status codes before touching the GPU."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "snapmla.h")
LIB = os.path.join(ROOT, "paper_2602_10718_amd", "libsnapmla.so")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(snapmla_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def sm():
    if not os.path.exists(LIB):
        pytest.fail("libsnapmla.so is not built (run __graft_entry__.build())")
    from paper_2602_10718_amd import snapmla
    return snapmla


def test_every_declared_symbol_is_exported(sm):
    names = _declared()
    assert len(names) >= 8
    lib = ctypes.CDLL(LIB)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in snapmla.h but not exported"
    assert set(names) == set(sm.EXPORTS)


def test_abi_version(sm):
    assert sm.snapmla_abi_version() == 3


def test_spin_limit_hook_validates(sm):
    assert sm.lib.snapmla_debug_set_spin_limit(-1) == 1
    assert sm.lib.snapmla_debug_set_spin_limit(1 << 22) == 0


def test_workspace_size_layout(sm):
    a = sm.snapmla_decode_workspace_size(64, 1, 64, 256, 0)
    b = sm.snapmla_decode_workspace_size(64, 1, 64, 256, 4096)
    assert a > 64 * 64 * (512 + 4) and b > a
    # partial outputs dominate: (parts + B) x 64 rows x 512 floats
    assert a >= (256 + 64) * 64 * 512 * 4


@pytest.mark.parametrize("args,status", [
    ((-1, 1, 64, 8, 0), 1),      # B < 0
    ((4, 3, 64, 8, 0), 1),       # q_len not in {1, 2}
    ((4, 1, 0, 8, 0), 1),        # H < 1
    ((4, 2, 129, 8, 0), 1),      # q_len*H > 256
    ((4, 1, 64, 0, 0), 1),       # num_splits < 1
    ((4, 1, 64, 8, 100), 1),     # chunk not a multiple of 64
])
def test_workspace_size_rejects(sm, args, status):
    out = ctypes.c_size_t(0)
    assert sm.lib.snapmla_decode_workspace_size(*args, ctypes.byref(out)) == status
    assert sm.snapmla_get_last_error() != ""


def test_decode_argument_errors_before_any_launch(sm):
    L = sm.lib
    # unsupported page size
    st = L.snapmla_decode(None, None, None, None, None, None, None, 2, 1, 16, 4, 8, 32, 0.1, 0, 8, 0, 0, None, 0, None, 0, None, None)
    assert st == 2
    # bad softmax scale
    st = L.snapmla_decode(None, None, None, None, None, None, None, 2, 1, 16, 4, 8, 64, float("nan"), 0, 8, 0, 0, None, 0, None, 0, None,
                          None)
    assert st == 1
    # null pointers
    st = L.snapmla_decode(None, None, None, None, None, None, None, 2, 1, 16, 4, 8, 64, 0.1, 0, 8, 0, 0, None, 0, None, 0, None, None)
    assert st == 1 and "null" in sm.snapmla_get_last_error()
    # misaligned pointer (never dereferenced: validation fails first)
    p = 16 * 1024 + 8
    st = L.snapmla_decode(p, p, p, p, p, 4096, 4096, 2, 1, 16, 4, 8, 64, 0.1, 0, 8, 0, 0, 4096, 1 << 30, None, 0, None, None)
    assert st == 4
    # workspace too small
    st = L.snapmla_decode(4096, 4096, 4096, 4096, 4096, 4096, 4096, 2, 1, 16, 4, 8, 64, 0.1, 0, 8, 0, 0, 4096, 16, None, 0, None, None)
    assert st == 3
    # causal flag
    st = L.snapmla_decode(4096, 4096, 4096, 4096, 4096, 4096, 4096, 2, 1, 16, 4, 8, 64, 0.1, 7, 8, 0, 0, 4096, 1 << 30, None, 0, None,
                          None)
    assert st == 1
    # unknown decode flags
    st = L.snapmla_decode(4096, 4096, 4096, 4096, 4096, 4096, 4096, 2, 1, 16, 4, 8, 64, 0.1, 0, 8, 0, 2, 4096,
                          1 << 30, None, 0, None, None)
    assert st == 1 and "flags" in sm.snapmla_get_last_error()
    # out_dtype out of range; lse without out; misaligned out
    st = L.snapmla_decode(4096, 4096, 4096, 4096, 4096, 4096, 4096, 2, 1, 16, 4, 8, 64, 0.1, 0, 8, 0, 0, 4096,
                          1 << 30, 4096, 2, None, None)
    assert st == 1 and "out_dtype" in sm.snapmla_get_last_error()
    st = L.snapmla_decode(4096, 4096, 4096, 4096, 4096, 4096, 4096, 2, 1, 16, 4, 8, 64, 0.1, 0, 8, 0, 0, 4096,
                          1 << 30, None, 0, 4096, None)
    assert st == 1 and "lse" in sm.snapmla_get_last_error()
    st = L.snapmla_decode(4096, 4096, 4096, 4096, 4096, 4096, 4096, 2, 1, 16, 4, 8, 64, 0.1, 0, 8, 0, 0, 4096,
                          1 << 30, 4104, 0, 4096, None)
    assert st == 4
    # empty batch is a no-op
    assert L.snapmla_decode(None, None, None, None, None, None, None, 0, 1, 16, 4, 8, 64, 0.1, 0, 8, 0, 0, None, 0, None, 0, None,
                            None) == 0


def test_decode_kernel_alone_refuses_an_unprepared_workspace(sm):
    """snapmla_debug_decode_kernel reads the start descriptors a preparation launch wrote; a workspace
    that no FP8 decode call with the same buffers and sizes prepared is refused on the host, before any
    launch (the pointers below are never dereferenced)."""
    L = sm.lib
    st = L.snapmla_debug_decode_kernel(4096, 4096, 4096, 4096, 4096, 4096, 4096, 2, 1, 16, 4, 8, 64, 0.1, 0, 8, 0, 0,
                                       4096, 1 << 30, None, 0, None, None)
    assert st == 1 and "not prepared" in sm.snapmla_get_last_error()
    # the ordinary argument checks still come first
    st = L.snapmla_debug_decode_kernel(4096, 4096, 4096, 4096, 4096, 4096, 4096, 2, 1, 16, 4, 8, 64, 0.1, 0, 8, 0, 0,
                                       4096, 16, None, 0, None, None)
    assert st == 3


def test_other_entry_points_validate(sm):
    L = sm.lib
    assert L.snapmla_quantize_append(None, None, None, None, 1, 1, 4, 4, 32, None, None, None, None) == 2
    assert L.snapmla_quantize_append(None, None, None, None, -1, 1, 4, 4, 64, None, None, None, None) == 1
    assert L.snapmla_quantize_append(None, None, None, None, 0, 1, 4, 4, 64, None, None, None, None) == 0
    assert L.snapmla_quantize_append(None, None, None, None, 2, 1, 4, 4, 64, None, None, None, None) == 1
    assert L.snapmla_quantize_rows(None, -1, None, None, None) == 1
    assert L.snapmla_quantize_rows(None, 0, None, None, None) == 0
    assert L.snapmla_quantize_rows(4100, 4, 4096, 4096, None) == 4
    assert L.snapmla_e4m3_encode(None, 5, None, None) == 1
    assert L.snapmla_combine(None, 0, None, 2, 1, 16, 8, 0, None, 3, None, None) == 1
    assert L.snapmla_combine(4096, 16, 4096, 2, 1, 16, 8, 0, 4096, 0, None, None) == 3


def test_fetch_dequant_validates(sm):
    L = sm.lib
    assert L.snapmla_fetch_dequant(None, None, None, None, None, 1, 4, 4, 32, None, None) == 2    # page size
    assert L.snapmla_fetch_dequant(None, None, None, None, None, -1, 4, 4, 64, None, None) == 1   # B < 0
    assert L.snapmla_fetch_dequant(None, None, None, None, None, 70000, 4, 4, 64, None, None) == 1
    assert L.snapmla_fetch_dequant(None, None, None, None, None, 2, 0, 4, 64, None, None) == 1    # max_pages
    assert L.snapmla_fetch_dequant(None, None, None, None, None, 0, 4, 4, 64, None, None) == 0    # nothing to do
    assert L.snapmla_fetch_dequant(None, None, None, None, None, 2, 4, 4, 64, None, None) == 1    # null pointers
    assert L.snapmla_fetch_dequant(4104, 4096, 4096, 4096, 4096, 2, 4, 4, 64, 4096, None) == 4   # misaligned latent
    assert L.snapmla_fetch_dequant(4096, 4096, 4096, 4098, 4096, 2, 4, 4, 64, 4096, None) == 4   # misaligned table


def test_bf16_entry_points_validate(sm):
    L = sm.lib
    # decode_bf16: same checks as snapmla_decode, no scale plane
    assert L.snapmla_decode_bf16(None, None, None, None, None, None, 2, 1, 16, 4, 8, 32, 0.1, 0, 8, 0, None, 0, None, 0, None,
                                 None) == 2                                                     # page size
    assert L.snapmla_decode_bf16(None, None, None, None, None, None, 2, 3, 16, 4, 8, 64, 0.1, 0, 8, 0, None, 0, None, 0, None,
                                 None) == 1                                                     # q_len
    assert L.snapmla_decode_bf16(None, None, None, None, None, None, 2, 1, 16, 4, 8, 64, 0.1, 0, 8, 0, None, 0, None, 0, None,
                                 None) == 1                                                     # null pointers
    assert L.snapmla_decode_bf16(4096, 4096, 4096, 4096, 4096, 4096, 2, 1, 16, 4, 8, 64, 0.1, 0, 8, 0, 4096, 16, None, 0, None,
                                 None) == 3                                                     # workspace
    assert L.snapmla_decode_bf16(4096, 4096, 4104, 4096, 4096, 4096, 2, 1, 16, 4, 8, 64, 0.1, 0, 8, 0, 4096,
                                 1 << 30, None, 0, None, None) == 4                                            # misaligned cache
    assert L.snapmla_decode_bf16(None, None, None, None, None, None, 0, 1, 16, 4, 8, 64, 0.1, 0, 8, 0, None, 0, None, 0, None,
                                 None) == 0                                                     # B == 0
    # append_bf16
    assert L.snapmla_append_bf16(None, None, None, None, 1, 1, 4, 4, 32, None, None, None) == 2
    assert L.snapmla_append_bf16(None, None, None, None, -1, 1, 4, 4, 64, None, None, None) == 1
    assert L.snapmla_append_bf16(None, None, None, None, 0, 1, 4, 4, 64, None, None, None) == 0
    assert L.snapmla_append_bf16(None, None, None, None, 2, 1, 4, 4, 64, None, None, None) == 1
    assert L.snapmla_append_bf16(4096, 4096, 4096, 4096, 2, 1, 4, 4, 64, 4100, 4096, None) == 4


def test_read_ceiling_validates(sm):
    L = sm.lib
    assert L.snapmla_debug_read_ceiling(None, None, None, None, -1, 4, 1, None, None) == 1        # nblk < 0
    assert L.snapmla_debug_read_ceiling(None, None, None, None, 10, 4, 0, None, None) == 1        # units < 1
    assert L.snapmla_debug_read_ceiling(None, None, None, None, 10, 0, 1, None, None) == 1        # num_pages < 1
    assert L.snapmla_debug_read_ceiling(4096, 4096, 4096, 4096, 1793, 4, 1, 4096, None) == 1      # > 1792 per unit
    assert L.snapmla_debug_read_ceiling(None, None, None, None, 10, 4, 1, 4096, None) == 1        # null pointers
    assert L.snapmla_debug_read_ceiling(4104, 4096, 4096, 4096, 10, 4, 1, 4096, None) == 4        # misaligned plane
    assert L.snapmla_debug_read_ceiling(4096, 4096, 4096, 4098, 10, 4, 1, 4096, None) == 4        # misaligned pages


def test_read_stream_validates(sm):
    L = sm.lib
    assert L.snapmla_debug_read_stream(4096, -16, 4, 4096, None) == 1        # bytes < 0
    assert L.snapmla_debug_read_stream(4096, 24, 4, 4096, None) == 1         # not a multiple of 16
    assert L.snapmla_debug_read_stream(4096, 64, 0, 4096, None) == 1         # grid < 1
    assert L.snapmla_debug_read_stream(None, 64, 4, 4096, None) == 1         # null buffer
    assert L.snapmla_debug_read_stream(4096, 64, 4, None, None) == 1         # null out
    assert L.snapmla_debug_read_stream(4104, 64, 4, 4096, None) == 4         # misaligned buffer
    assert L.snapmla_debug_read_stream(4096, 64, 4, 4098, None) == 4         # misaligned out



def test_append_decode_validates(sm):
    L = sm.lib
    big = 1 << 30
    # n_new < 0; then the decode's own checks (q_len 3); then null / misaligned new-token pointers
    assert L.snapmla_append_decode(None, None, -1, 4096, 4096, 4096, 4096, 4096, 4096, 4096, 2, 1, 16, 4, 8, 64,
                                   0.1, 0, 8, 0, 0, 4096, big, None, 0, None, None) == 1
    assert L.snapmla_append_decode(4096, 4096, 1, 4096, 4096, 4096, 4096, 4096, 4096, 4096, 2, 3, 16, 4, 8, 64,
                                   0.1, 0, 8, 0, 0, 4096, big, None, 0, None, None) == 1
    assert L.snapmla_append_decode(None, 4096, 1, 4096, 4096, 4096, 4096, 4096, 4096, 4096, 2, 1, 16, 4, 8, 64,
                                   0.1, 0, 8, 0, 0, 4096, big, None, 0, None, None) == 1
    assert L.snapmla_append_decode(4104, 4096, 1, 4096, 4096, 4096, 4096, 4096, 4096, 4096, 2, 1, 16, 4, 8, 64,
                                   0.1, 0, 8, 0, 0, 4096, big, None, 0, None, None) == 4
    assert L.snapmla_append_decode(None, None, 1, None, None, None, None, None, None, None, 0, 1, 16, 4, 8, 64,
                                   0.1, 0, 8, 0, 0, None, 0, None, 0, None, None) == 0                            # B == 0
