"""Device-side staging for a decode workload: cache planes, queries, workspace, and one step.

A step is the whole hot path for one batch: quantize-and-append the step's new
tokens, quantize the queries and decode (one snapmla_append_decode call: the
append runs in the decode's preparation launch), and merge the KV pieces
(snapmla_combine).  Everything runs in libsnapmla.so; torch only owns
the device buffers and the stream.
"""

import numpy as np
import torch

from . import snapmla as sm
from .workloads import D_C, D_R, PAGE


def _dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype) if dtype is not None \
        else torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _u16_to_bf16(a):
    """uint16 bit patterns (numpy) -> torch bfloat16 on the device, bit for bit."""
    t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()
    return t.view(torch.bfloat16)


# A period (one 64-token block) of a decode workgroup takes ~2 us; a combine launch
# costs about as much as four of them on a small batch (measured on 1 x 256 tokens:
# 27.4 us per step with 8 parts + combine, 21.7 us with one piece and no combine).
UNSPLIT_SLACK_BLOCKS = 4


def prefer_unsplit(seq_lens, q_len, H, kv_dtype="e4m3", device=None):
    """Whether the unsplit plan (one piece per sequence, rows written by the decode, no combine) is
    expected to be faster than the balanced split + combine: every sequence's workgroups fit on the
    chip at once, the longest sequence holds at most UNSPLIT_SLACK_BLOCKS more blocks than a part of
    the balanced plan, and the decode writes direct rows for this shape (the FP8-cache decode with one
    64-row group, the BF16-cache decode always)."""
    groups = (q_len * H + 63) // 64
    if kv_dtype != "bf16" and groups > 1:
        return False
    props = torch.cuda.get_device_properties(device if device is not None else torch.cuda.current_device())
    blocks = (np.asarray(seq_lens, np.int64) + PAGE - 1) // PAGE
    if len(blocks) == 0 or len(blocks) * groups > props.multi_processor_count:
        return False
    parts = sm.default_num_splits(q_len, H, device=device, total_blocks=int(blocks.sum()))
    return int(blocks.max()) <= blocks.sum() / parts + UNSPLIT_SLACK_BLOCKS


class DecodeRunner:
    """Holds one workload's device buffers.

    The cache is filled with snapmla_quantize_append (all tokens before the
    step's n_new); step() appends the n_new step tokens, decodes and combines.
    """

    def __init__(self, wl, num_splits=None, kv_chunk_tokens=None, out_dtype=torch.float32, fill=True, cache=None,
                 kv_dtype="e4m3", exact_qk=False, direct=True, unsplit=False):
        """cache: (kv_latent, kv_scale, k_rope) of another runner over the same sequences, pages and
        tokens, used instead of allocating and filling a new one.  kv_dtype "bf16": a BF16 cache
        (kv_latent bf16, no scales) written by snapmla_append_bf16 and read by snapmla_decode_bf16.
        exact_qk: decode with SNAPMLA_DECODE_EXACT_QK (content term accumulated exactly in float32).
        direct: the decode writes the rows of sequences that one piece covers into out/lse itself
        (False: partials only, every row from the combine).  unsplit: one piece per sequence (fixed
        chunks as long as the page table, one split), so that the step needs no combine; "auto": that plan
        when prefer_unsplit expects it to be faster and no plan is given."""
        self.kv_dtype = kv_dtype
        self.flags = sm.DECODE_EXACT_QK if exact_qk else 0
        self.wl = wl
        self.B, self.H, self.q_len = wl.B, wl.H, wl.q_len
        self.direct = direct
        if unsplit == "auto":
            unsplit = num_splits is None and kv_chunk_tokens is None and wl.kv_chunk_tokens == 0 and \
                prefer_unsplit(wl.seq_lens, wl.q_len, wl.H, kv_dtype)
        if unsplit:
            kv_chunk_tokens, num_splits = wl.max_pages * PAGE, 1
        self.kv_chunk_tokens = wl.kv_chunk_tokens if kv_chunk_tokens is None else kv_chunk_tokens
        if num_splits is None:
            if self.kv_chunk_tokens > 0:
                num_splits = max(1, int(np.max((wl.seq_lens + self.kv_chunk_tokens - 1) // self.kv_chunk_tokens)))
            else:
                num_splits = sm.default_num_splits(self.q_len, self.H,
                                                   total_blocks=int(((wl.seq_lens.astype(np.int64) + 63) // 64).sum()))
        self.num_splits = num_splits
        # with fixed chunks as long as the page table and one split, no sequence is split: the decode
        # writes every row (direct) and the combine has nothing to do
        # (the FP8-cache decode writes direct rows with one 64-row group; the BF16-cache decode always)
        direct_rows = direct and (kv_dtype == "bf16" or self.q_len * self.H <= 64)
        self.needs_combine = not (direct_rows and self.kv_chunk_tokens >= wl.max_pages * PAGE and num_splits == 1)
        P = wl.num_pages
        if cache is not None:
            self.kv_latent, self.kv_scale, self.k_rope = cache
            fill = False
        elif kv_dtype == "bf16":
            self.kv_latent = torch.zeros((P, PAGE, D_C), dtype=torch.bfloat16, device="cuda")
            self.kv_scale = None
            self.k_rope = torch.zeros((P, PAGE, D_R), dtype=torch.bfloat16, device="cuda")
        else:
            self.kv_latent = torch.zeros((P, PAGE, D_C), dtype=torch.uint8, device="cuda")
            self.kv_scale = torch.zeros((P, PAGE), dtype=torch.float32, device="cuda")
            self.k_rope = torch.zeros((P, PAGE, D_R), dtype=torch.bfloat16, device="cuda")
        self.page_table = _dev(wl.page_table, torch.int32)
        self.seq_lens = _dev(wl.seq_lens, torch.int32)
        qn, qr = wl.queries()
        self.q_nope = _u16_to_bf16(qn)
        self.q_rope = _u16_to_bf16(qr)
        ws = sm.snapmla_decode_workspace_size(self.B, self.q_len, self.H, self.num_splits, self.kv_chunk_tokens)
        self.workspace = torch.empty(ws, dtype=torch.uint8, device="cuda")
        self.out = torch.empty((self.B, self.q_len, self.H, D_C), dtype=out_dtype, device="cuda")
        self.lse = torch.empty((self.B, self.q_len, self.H), dtype=torch.float32, device="cuda")
        # the step's new tokens (the last n_new of every sequence)
        n_new = wl.n_new
        ck = np.zeros((self.B, n_new, D_C), np.uint16)
        kr = np.zeros((self.B, n_new, D_R), np.uint16)
        for b in range(self.B):
            N = int(wl.seq_lens[b])
            lo = max(0, N - n_new)              # new token t lands at position N - n_new + t
            if N > lo:
                ck[b, lo - (N - n_new):], kr[b, lo - (N - n_new):] = wl.tokens(b, lo, N)
        self.new_ckv = _u16_to_bf16(ck)
        self.new_krope = _u16_to_bf16(kr)
        if fill:
            self.fill_prefix()

    def fill_prefix(self, chunk=16384):
        """Append every sequence's tokens before the step's new ones, in bulk."""
        wl = self.wl
        for b in range(self.B):
            N = int(wl.seq_lens[b]) - wl.n_new
            for t0 in range(0, max(N, 0), chunk):
                t1 = min(N, t0 + chunk)
                ck, kr = wl.tokens(b, t0, t1)
                pt = self.page_table[b:b + 1].clone()
                sl = torch.tensor([t1], dtype=torch.int32, device="cuda")
                if self.kv_dtype == "bf16":
                    sm.snapmla_append_bf16(_u16_to_bf16(ck[None]), _u16_to_bf16(kr[None]), pt, sl, wl.num_pages,
                                           self.kv_latent, self.k_rope)
                else:
                    sm.snapmla_quantize_append(_u16_to_bf16(ck[None]), _u16_to_bf16(kr[None]), pt, sl,
                                               wl.num_pages, self.kv_latent, self.kv_scale, self.k_rope)
        torch.cuda.synchronize()

    def append(self, stream=None):
        if self.kv_dtype == "bf16":
            sm.snapmla_append_bf16(self.new_ckv, self.new_krope, self.page_table, self.seq_lens, self.wl.num_pages,
                                   self.kv_latent, self.k_rope, stream=stream)
            return
        sm.snapmla_quantize_append(self.new_ckv, self.new_krope, self.page_table, self.seq_lens, self.wl.num_pages,
                                   self.kv_latent, self.kv_scale, self.k_rope, stream=stream)

    def _out(self):
        return (self.out, self.lse) if self.direct else (None, None)

    def decode(self, stream=None):
        out, lse = self._out()
        if self.kv_dtype == "bf16":
            sm.snapmla_decode_bf16(self.q_nope, self.q_rope, self.kv_latent, self.k_rope, self.page_table,
                                   self.seq_lens, self.wl.tau, self.wl.causal, self.num_splits,
                                   self.kv_chunk_tokens, self.workspace, stream=stream, out=out, lse=lse)
            return
        sm.snapmla_decode(self.q_nope, self.q_rope, self.kv_latent, self.kv_scale, self.k_rope, self.page_table,
                          self.seq_lens, self.wl.tau, self.wl.causal, self.num_splits, self.kv_chunk_tokens,
                          self.workspace, stream=stream, flags=self.flags, out=out, lse=lse)

    def decode_kernel_only(self, stream=None):
        """Measurement only: the decode launch of decode() alone, over the workspace the last decode() or
        append_decode() prepared (FP8 cache)."""
        out, lse = self._out()
        sm.snapmla_debug_decode_kernel(self.q_nope, self.q_rope, self.kv_latent, self.kv_scale, self.k_rope,
                                       self.page_table, self.seq_lens, self.wl.tau, self.wl.causal, self.num_splits,
                                       self.kv_chunk_tokens, self.workspace, stream=stream, flags=self.flags, out=out,
                                       lse=lse)

    def combine(self, stream=None):
        sm.snapmla_combine(self.workspace, self.seq_lens, self.B, self.q_len, self.H, self.num_splits,
                           self.kv_chunk_tokens, self.out, self.lse, stream=stream)

    def append_decode(self, stream=None):
        """The step's append and decode in one call (the append runs in the decode's preparation launch)."""
        out, lse = self._out()
        sm.snapmla_append_decode(self.new_ckv, self.new_krope, self.q_nope, self.q_rope, self.kv_latent, self.kv_scale,
                                 self.k_rope, self.page_table, self.seq_lens, self.wl.tau, self.wl.causal,
                                 self.num_splits, self.kv_chunk_tokens, self.workspace, stream=stream,
                                 flags=self.flags, out=out, lse=lse)

    def step(self, stream=None):
        if self.kv_dtype == "bf16":
            self.append(stream)
            self.decode(stream)
        else:
            self.append_decode(stream)
        if self.needs_combine:
            self.combine(stream)

    def sequence_cache(self, b):
        """(codes uint8 [N, 512], scales f32 [N], rope bits uint16 [N, 64]) of sequence b read back via the page table;
        for a BF16 cache (latent bits uint16 [N, 512], None, rope bits)."""
        N = int(self.wl.seq_lens[b])
        npg = (N + PAGE - 1) // PAGE
        pages = self.page_table[b, :npg].long()
        if self.kv_dtype == "bf16":
            lat = self.kv_latent[pages].reshape(-1, D_C)[:N].view(torch.int16).cpu().numpy().view(np.uint16)
            rope = self.k_rope[pages].reshape(-1, D_R)[:N].view(torch.int16).cpu().numpy().view(np.uint16)
            return lat, None, rope
        codes = self.kv_latent[pages].reshape(-1, D_C)[:N].cpu().numpy()
        scales = self.kv_scale[pages].reshape(-1)[:N].cpu().numpy()
        rope = self.k_rope[pages].reshape(-1, D_R)[:N].view(torch.int16).cpu().numpy().view(np.uint16)
        return codes, scales, rope
