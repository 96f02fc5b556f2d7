"""ctypes binding of libsnapmla.so with the C function names (include/snapmla.h).

Argument marshalling only: every computation runs in the HIP library.  Device
buffers are torch tensors (used for allocation and streams); the current torch
stream is passed as the hipStream_t.  Importing this module loads the library
and raises if it has not been built.
"""

import ctypes
import math
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("SNAPMLA_LIB") or os.path.join(_HERE, "libsnapmla.so")

SNAPMLA_OK = 0
STATUS_NAMES = {0: "OK", 1: "INVALID_ARGUMENT", 2: "UNSUPPORTED", 3: "WORKSPACE_TOO_SMALL", 4: "MISALIGNED",
                5: "HIP_ERROR"}

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2602_10718_amd.build` "
                      "(or __graft_entry__.build())")

lib = ctypes.CDLL(LIB_PATH)

_p = ctypes.c_void_p
_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_f32 = ctypes.c_float
_sz = ctypes.c_size_t

lib.snapmla_abi_version.restype = ctypes.c_int
lib.snapmla_abi_version.argtypes = []
lib.snapmla_get_last_error.restype = ctypes.c_char_p
lib.snapmla_get_last_error.argtypes = []
lib.snapmla_quantize_append.restype = ctypes.c_int
lib.snapmla_quantize_append.argtypes = [_p, _p, _p, _p, _i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p]
lib.snapmla_quantize_rows.restype = ctypes.c_int
lib.snapmla_quantize_rows.argtypes = [_p, _i64, _p, _p, _p]
lib.snapmla_decode_workspace_size.restype = ctypes.c_int
lib.snapmla_decode_workspace_size.argtypes = [_i32, _i32, _i32, _i32, _i32, ctypes.POINTER(_sz)]
lib.snapmla_decode.restype = ctypes.c_int
lib.snapmla_decode.argtypes = [_p, _p, _p, _p, _p, _p, _p, _i32, _i32, _i32, _i32, _i32, _i32, _f32, _i32, _i32,
                               _i32, _i32, _p, _sz, _p, _i32, _p, _p]
lib.snapmla_debug_decode_kernel.restype = ctypes.c_int
lib.snapmla_debug_decode_kernel.argtypes = lib.snapmla_decode.argtypes
lib.snapmla_combine.restype = ctypes.c_int
lib.snapmla_combine.argtypes = [_p, _sz, _p, _i32, _i32, _i32, _i32, _i32, _p, _i32, _p, _p]
lib.snapmla_e4m3_encode.restype = ctypes.c_int
lib.snapmla_e4m3_encode.argtypes = [_p, _i64, _p, _p]
lib.snapmla_quantize_cache_config.restype = ctypes.c_int
lib.snapmla_quantize_cache_config.argtypes = [_p, _p, _p, _p, _i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _p]
lib.snapmla_decode_bf16.restype = ctypes.c_int
lib.snapmla_decode_bf16.argtypes = [_p, _p, _p, _p, _p, _p, _i32, _i32, _i32, _i32, _i32, _i32, _f32, _i32, _i32,
                                    _i32, _p, _sz, _p, _i32, _p, _p]
lib.snapmla_append_bf16.restype = ctypes.c_int
lib.snapmla_append_bf16.argtypes = [_p, _p, _p, _p, _i32, _i32, _i32, _i32, _i32, _p, _p, _p]
lib.snapmla_fetch_dequant.restype = ctypes.c_int
lib.snapmla_fetch_dequant.argtypes = [_p, _p, _p, _p, _p, _i32, _i32, _i32, _i32, _p, _p]
lib.snapmla_append_decode.restype = ctypes.c_int
lib.snapmla_append_decode.argtypes = [_p, _p, _i32, _p, _p, _p, _p, _p, _p, _p, _i32, _i32, _i32, _i32, _i32, _i32,
                                      _f32, _i32, _i32, _i32, _i32, _p, _sz, _p, _i32, _p, _p]
lib.snapmla_debug_read_ceiling.restype = ctypes.c_int
lib.snapmla_debug_mfma_fp8.restype = ctypes.c_int
lib.snapmla_debug_mfma_fp8.argtypes = [_p, _p, _p, _i64, _p]
lib.snapmla_debug_set_spin_limit.restype = ctypes.c_int
lib.snapmla_debug_set_spin_limit.argtypes = [_i32]
lib.snapmla_debug_read_ceiling.argtypes = [_p, _p, _p, _p, _i32, _i32, _i32, _p, _p]
lib.snapmla_append_decode_noalloc.restype = ctypes.c_int
lib.snapmla_append_decode_noalloc.argtypes = [_p, _p, _i32, _p, _p, _p, _p, _p, _p, _p, _i32, _i32, _i32, _i32, _i32,
                                              _i32, ctypes.c_float, _i32, _i32, _i32, _i32, _p, _i32, _p, _p]
lib.snapmla_debug_read_stream.restype = ctypes.c_int
lib.snapmla_debug_read_stream.argtypes = [_p, _i64, _i32, _p, _p]

EXPORTS = ["snapmla_abi_version", "snapmla_get_last_error", "snapmla_quantize_append", "snapmla_quantize_rows",
           "snapmla_decode_workspace_size", "snapmla_decode", "snapmla_combine", "snapmla_e4m3_encode",
           "snapmla_fetch_dequant", "snapmla_quantize_cache_config", "snapmla_decode_bf16", "snapmla_append_bf16",
           "snapmla_debug_read_ceiling", "snapmla_append_decode", "snapmla_debug_set_spin_limit",
           "snapmla_debug_mfma_fp8", "snapmla_debug_read_stream", "snapmla_append_decode_noalloc",
           "snapmla_debug_decode_kernel"]

CACHE_CONFIGS = {"snapmla": 0, "A": 1, "B": 2, "C": 3, "D": 4}


class SnapMLAError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"snapmla status {status} ({STATUS_NAMES.get(status, '?')}): {msg}")
        self.status = status


def _check(status):
    if status != SNAPMLA_OK:
        raise SnapMLAError(status, lib.snapmla_get_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("snapmla buffers must be device tensors")
    if not t.is_contiguous():
        raise ValueError("snapmla buffers must be contiguous")
    return t.data_ptr()


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def snapmla_abi_version():
    return lib.snapmla_abi_version()


def snapmla_get_last_error():
    return lib.snapmla_get_last_error().decode()


def snapmla_quantize_append(c_kv_new, k_rope_new, page_table, seq_lens, num_pages, kv_latent, kv_scale, k_rope,
                            page_size=64, stream=None):
    """c_kv_new bf16 [B, n_new, 512], k_rope_new bf16 [B, n_new, 64], page_table int32 [B, max_pages],
    seq_lens int32 [B]; writes into kv_latent uint8 [num_pages, 64, 512], kv_scale f32 [num_pages, 64],
    k_rope bf16 [num_pages, 64, 64]."""
    B, n_new = c_kv_new.shape[0], c_kv_new.shape[1]
    _check(lib.snapmla_quantize_append(_ptr(c_kv_new), _ptr(k_rope_new), _ptr(page_table), _ptr(seq_lens), B, n_new,
                                       page_table.shape[1], num_pages, page_size, _ptr(kv_latent), _ptr(kv_scale),
                                       _ptr(k_rope), _stream(stream)))


def snapmla_quantize_rows(x, codes, scale, stream=None):
    """x bf16 [rows, 512] -> codes uint8 [rows, 512], scale f32 [rows]."""
    _check(lib.snapmla_quantize_rows(_ptr(x), x.numel() // 512, _ptr(codes), _ptr(scale), _stream(stream)))


def snapmla_debug_read_stream(buf, grid, out, stream=None):
    """Measurement hook: read the whole of `buf` (a device tensor, 16-byte multiple) once with plain
    16-byte vector loads by `grid` workgroups; `out` int32 [grid] receives per-workgroup XOR checksums."""
    nbytes = buf.numel() * buf.element_size()
    _check(lib.snapmla_debug_read_stream(_ptr(buf), nbytes, grid, _ptr(out), _stream(stream)))


def snapmla_debug_read_ceiling(kv_latent, kv_scale, k_rope, pages, num_pages, units, out, stream=None):
    """Measurement hook: stream the cache pages listed in `pages` (int32 [nblk], stream order) into LDS
    through the decode's copy structure, with no attention arithmetic; `out` uint32-sized int32 [units]
    receives per-unit checksums (XOR of the first KiB of every latent and RoPE page of the unit)."""
    _check(lib.snapmla_debug_read_ceiling(_ptr(kv_latent), _ptr(kv_scale), _ptr(k_rope), _ptr(pages), pages.numel(),
                                          num_pages, units, _ptr(out), _stream(stream)))


def snapmla_e4m3_encode(x, codes, stream=None):
    _check(lib.snapmla_e4m3_encode(_ptr(x), x.numel(), _ptr(codes), _stream(stream)))


def snapmla_decode_workspace_size(B, q_len, H, num_splits, kv_chunk_tokens):
    out = _sz(0)
    _check(lib.snapmla_decode_workspace_size(B, q_len, H, num_splits, kv_chunk_tokens, ctypes.byref(out)))
    return out.value


DECODE_EXACT_QK = 1   # snapmla_decode_flags: content term with exact float32 accumulation


def _out_args(out, lse):
    """(out pointer, out_dtype, lse pointer) of the decode calls; out None: partials only."""
    if out is None:
        if lse is not None:
            raise ValueError("lse without out")
        return None, 0, None
    return _ptr(out), _out_dtype(out), _ptr(lse)


def snapmla_decode(q_nope, q_rope, kv_latent, kv_scale, k_rope, page_table, seq_lens, softmax_scale, causal,
                   num_splits, kv_chunk_tokens, workspace, page_size=64, stream=None, flags=0, out=None, lse=None):
    """q_nope bf16 [B, q_len, H, 512], q_rope bf16 [B, q_len, H, 64]; cache planes as in snapmla_quantize_append;
    workspace uint8 of at least snapmla_decode_workspace_size(...) bytes; flags 0 or DECODE_EXACT_QK.
    out bf16 or f32 [B, q_len, H, 512] and lse f32 [B, q_len, H] (or None): the rows of sequences that one
    piece covers are written here directly, the others by snapmla_combine with the same out/lse."""
    B, q_len, H = q_nope.shape[0], q_nope.shape[1], q_nope.shape[2]
    _check(lib.snapmla_decode(_ptr(q_nope), _ptr(q_rope), _ptr(kv_latent), _ptr(kv_scale), _ptr(k_rope),
                              _ptr(page_table), _ptr(seq_lens), B, q_len, H, page_table.shape[1], kv_latent.shape[0],
                              page_size, float(softmax_scale), int(causal), num_splits, kv_chunk_tokens, int(flags),
                              _ptr(workspace), workspace.numel() * workspace.element_size(), *_out_args(out, lse),
                              _stream(stream)))


def snapmla_debug_decode_kernel(q_nope, q_rope, kv_latent, kv_scale, k_rope, page_table, seq_lens, softmax_scale,
                                causal, num_splits, kv_chunk_tokens, workspace, page_size=64, stream=None, flags=0,
                                out=None, lse=None):
    """Measurement only: snapmla_decode's decode launch alone, over a workspace that a snapmla_decode (or
    snapmla_append_decode) call with the same arguments prepared on the same stream (a workspace that no
    matching FP8 call prepared last is refused with SnapMLAError)."""
    B, q_len, H = q_nope.shape[0], q_nope.shape[1], q_nope.shape[2]
    _check(lib.snapmla_debug_decode_kernel(_ptr(q_nope), _ptr(q_rope), _ptr(kv_latent), _ptr(kv_scale), _ptr(k_rope),
                                           _ptr(page_table), _ptr(seq_lens), B, q_len, H, page_table.shape[1],
                                           kv_latent.shape[0], page_size, float(softmax_scale), int(causal), num_splits,
                                           kv_chunk_tokens, int(flags), _ptr(workspace),
                                           workspace.numel() * workspace.element_size(), *_out_args(out, lse),
                                           _stream(stream)))


def snapmla_append_decode(c_kv_new, k_rope_new, q_nope, q_rope, kv_latent, kv_scale, k_rope, page_table, seq_lens,
                          softmax_scale, causal, num_splits, kv_chunk_tokens, workspace, page_size=64, stream=None,
                          flags=0, out=None, lse=None):
    """snapmla_quantize_append of c_kv_new bf16 [B, n_new, 512] / k_rope_new bf16 [B, n_new, 64] followed by
    snapmla_decode (out, lse as there), the append run in the decode's preparation launch."""
    B, q_len, H = q_nope.shape[0], q_nope.shape[1], q_nope.shape[2]
    n_new = c_kv_new.shape[1]
    _check(lib.snapmla_append_decode(_ptr(c_kv_new), _ptr(k_rope_new), n_new, _ptr(q_nope), _ptr(q_rope),
                                     _ptr(kv_latent), _ptr(kv_scale), _ptr(k_rope), _ptr(page_table), _ptr(seq_lens),
                                     B, q_len, H, page_table.shape[1], kv_latent.shape[0], page_size,
                                     float(softmax_scale), int(causal), num_splits, kv_chunk_tokens, int(flags),
                                     _ptr(workspace), workspace.numel() * workspace.element_size(),
                                     *_out_args(out, lse), _stream(stream)))


NOALLOC_SCRATCH_BYTES = 128 << 20   # SNAPMLA_NOALLOC_SCRATCH_BYTES


def snapmla_append_decode_noalloc(c_kv_new, k_rope_new, q_nope, q_rope, kv_latent, kv_scale, k_rope, page_table,
                                  seq_lens, softmax_scale, causal, num_splits, kv_chunk_tokens, out, lse=None,
                                  page_size=64, stream=None, flags=0):
    """snapmla_append_decode + snapmla_combine with the workspace in the library's static scratch (for callers
    that cannot allocate); out bf16 or f32 [B, q_len, H, 512], lse f32 [B, q_len, H] or None."""
    B, q_len, H = q_nope.shape[0], q_nope.shape[1], q_nope.shape[2]
    n_new = c_kv_new.shape[1]
    _check(lib.snapmla_append_decode_noalloc(_ptr(c_kv_new), _ptr(k_rope_new), n_new, _ptr(q_nope), _ptr(q_rope),
                                             _ptr(kv_latent), _ptr(kv_scale), _ptr(k_rope), _ptr(page_table),
                                             _ptr(seq_lens), B, q_len, H, page_table.shape[1], kv_latent.shape[0],
                                             page_size, float(softmax_scale), int(causal), num_splits,
                                             kv_chunk_tokens, int(flags), _ptr(out), _out_dtype(out), _ptr(lse),
                                             _stream(stream)))


def _out_dtype(out):
    if out.dtype == torch.float32:
        return 1
    if out.dtype == torch.bfloat16:
        return 0
    raise ValueError("out must be bfloat16 or float32")


def snapmla_combine(workspace, seq_lens, B, q_len, H, num_splits, kv_chunk_tokens, out, lse=None, stream=None):
    """out bf16 or f32 [B, q_len, H, 512]; lse f32 [B, q_len, H] or None."""
    if out.dtype == torch.float32:
        od = 1
    elif out.dtype == torch.bfloat16:
        od = 0
    else:
        raise ValueError("out must be bfloat16 or float32")
    _check(lib.snapmla_combine(_ptr(workspace), workspace.numel() * workspace.element_size(), _ptr(seq_lens), B,
                               q_len, H, num_splits, kv_chunk_tokens, _ptr(out), od, _ptr(lse), _stream(stream)))


def default_num_splits(q_len, H, device=None, total_blocks=None):
    """One workgroup per compute unit across all row groups, rounded down to a multiple of 8; with
    total_blocks (the batch's 64-token blocks) given, no more parts than blocks (rounded up to a
    multiple of 8), so that a small batch launches no idle parts for the combine to step over."""
    props = torch.cuda.get_device_properties(device if device is not None else torch.cuda.current_device())
    groups = math.ceil(q_len * H / 64)
    n = max(8, (props.multi_processor_count // groups) // 8 * 8)
    if total_blocks is not None:
        n = min(n, max(8, (int(total_blocks) + 7) // 8 * 8))
    return n


def snapmla_fetch_dequant(kv_latent, kv_scale, k_rope, page_table, cu_seqlens, out, page_size=64, stream=None):
    """cu_seqlens int32 [B+1] (device); out bf16 [cu_seqlens[B], 576]: per cached token the dequantized
    latent (512) then the RoPE key (64)."""
    B = cu_seqlens.numel() - 1
    _check(lib.snapmla_fetch_dequant(_ptr(kv_latent), _ptr(kv_scale), _ptr(k_rope), _ptr(page_table),
                                     _ptr(cu_seqlens), B, page_table.shape[1], kv_latent.shape[0], page_size,
                                     _ptr(out), _stream(stream)))


def snapmla_quantize_cache_config(c_kv, k_rope, page_table, cu_seqlens, config, kv_latent, kv_scale, k_rope_out,
                                  scratch=None, page_size=64, stream=None):
    """c_kv bf16 [T, 512], k_rope bf16 [T, 64] (token j of sequence b at row cu_seqlens[b] + j); config one of
    CACHE_CONFIGS' names or numbers; scratch: int32 device tensor of >= 1 element (needed for config "C")."""
    cfg = CACHE_CONFIGS[config] if isinstance(config, str) else int(config)
    B = cu_seqlens.numel() - 1
    _check(lib.snapmla_quantize_cache_config(_ptr(c_kv), _ptr(k_rope), _ptr(page_table), _ptr(cu_seqlens), B,
                                             page_table.shape[1], kv_latent.shape[0], page_size, cfg, _ptr(scratch),
                                             _ptr(kv_latent), _ptr(kv_scale), _ptr(k_rope_out), _stream(stream)))


def snapmla_decode_bf16(q_nope, q_rope, kv_latent, k_rope, page_table, seq_lens, softmax_scale, causal, num_splits,
                        kv_chunk_tokens, workspace, page_size=64, stream=None, out=None, lse=None):
    """kv_latent bf16 [num_pages, 64, 512]; otherwise as snapmla_decode (without kv_scale)."""
    B, q_len, H = q_nope.shape[0], q_nope.shape[1], q_nope.shape[2]
    _check(lib.snapmla_decode_bf16(_ptr(q_nope), _ptr(q_rope), _ptr(kv_latent), _ptr(k_rope), _ptr(page_table),
                                   _ptr(seq_lens), B, q_len, H, page_table.shape[1], kv_latent.shape[0], page_size,
                                   float(softmax_scale), int(causal), num_splits, kv_chunk_tokens, _ptr(workspace),
                                   workspace.numel() * workspace.element_size(), *_out_args(out, lse),
                                   _stream(stream)))


def snapmla_append_bf16(c_kv_new, k_rope_new, page_table, seq_lens, num_pages, kv_latent, k_rope, page_size=64,
                        stream=None):
    """c_kv_new bf16 [B, n_new, 512], k_rope_new bf16 [B, n_new, 64] into kv_latent bf16 [num_pages, 64, 512]."""
    B, n_new = c_kv_new.shape[0], c_kv_new.shape[1]
    _check(lib.snapmla_append_bf16(_ptr(c_kv_new), _ptr(k_rope_new), _ptr(page_table), _ptr(seq_lens), B, n_new,
                                   page_table.shape[1], num_pages, page_size, _ptr(kv_latent), _ptr(k_rope),
                                   _stream(stream)))


def snapmla_debug_set_spin_limit(polls):
    """Bound on the polls of every handshake wait in later decode calls (test hook; see include/snapmla.h)."""
    _check(lib.snapmla_debug_set_spin_limit(int(polls)))


def snapmla_debug_mfma_fp8(a, b, c, stream=None):
    """a, b uint8 [tiles, 16, 128] E4M3 codes; c float32 [tiles, 16, 16] = one FP8 MFMA per tile."""
    _check(lib.snapmla_debug_mfma_fp8(_ptr(a), _ptr(b), _ptr(c), a.shape[0], _stream(stream)))
