"""Benchmark of the SnapMLA FP8 MLA decode hot path on one MI355X.

One step = the whole hot path for one batch: quantize-and-append the step's new
tokens into the paged FP8 cache (snapmla_quantize_append), quantize the queries
and decode every sequence (snapmla_decode: FP8 QK + BF16 RoPE, online softmax,
fused and block-quantized P, FP8 PV), and merge the split-KV pieces
(snapmla_combine; skipped under the unsplit plan, where the decode writes every
row itself -- the plan bench.py picks for small batches, --plan).  Inputs are
resident in HBM before timing starts.

Default workload: 64-head MLA decode, batch 64, one query token, ragged context
lengths uniform in [8192, 32768], 64-token pages in shuffled physical order.

`value` is the achieved KV-cache read rate, sum of context lengths x 644 B per
token / step time, over K back-to-back steps after W warm-up steps, with the QK
content term on the FP8 matrix cores (the default mode).  Also reported: the
same step in the exact-accumulation QK mode (SNAPMLA_DECODE_EXACT_QK) on the same
cache; the step captured once as a HIP graph and replayed; cold-cache step times
(a 1 GiB scratch write and read between steps, outside the timed region: the
read leaves the caches clean, so no write-back of scratch lines lands inside the
step); the per-call split; the roofline of the decode call, with two measured
reference rates beside the 8 TB/s peak (the decode's own copy structure without
arithmetic, and a plain 16-byte-load read stream over as many bytes); the error
of both QK modes against an unquantized reference (fp32 attention on the bf16
inputs) on sampled sequences; and the CPU oracle on a bounded sample.

Prints ONE JSON line on stdout; progress goes to stderr.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MLA decode µs/step + achieved KV HBM GB/s (% of peak), 64 heads, 32K ctx"
HBM_PEAK_GBPS = 8000.0
BYTES_PER_TOKEN = 512 + 2 * 64 + 4           # e4m3 latent + bf16 rope + f32 scale
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "decode_traffic.json")


def _log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


SOURCES_OF = {"decode": ("decode.hip", "quant.hip", "piece_end.h", "snapmla_device.h", "snapmla_internal.h"),
              "fetch_dequant": ("fetch.hip", "snapmla_device.h"),
              "decode_bf16": ("decode_bf16.hip", "quant.hip", "piece_end.h", "snapmla_device.h",
                              "snapmla_internal.h")}


def _src_hash(op="decode"):
    h = hashlib.sha256()
    for f in SOURCES_OF[op]:
        h.update(open(os.path.join(ROOT, "paper_2602_10718_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def _traffic(key, op="decode", kernel=None):
    """HBM bytes per launch measured with rocprofv3 counters (profiles/), if the sources still match: of the
    whole call, or of one of its kernels (read + written)."""
    try:
        d = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    e = d.get(key)
    if not e or e.get("src_hash") != _src_hash(op):
        return None
    if kernel is not None:
        k = e.get(kernel)
        return None if not k else k["read"] + k["write"]
    return e.get("hbm_bytes_per_launch")


def cpu_baseline(w, budget_s=15.0):
    """The oracle (float64 numpy, as written) on a bounded sample of the same workload."""
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = 1
    from oracle import mla, quant
    qn, qr = w.queries()
    el = 0.0          # oracle compute time only (input generation excluded)
    toks = 0
    seqs = 0
    for b in range(w.B):
        N = int(w.seq_lens[b])
        ck, kr = w.tokens(b, 0, N)
        ts = time.perf_counter()
        q8, sq = quant.quantize_rows(qn[b].reshape(-1, 512))
        c8, sk = quant.quantize_rows(ck)
        vis = mla.visible_counts(N, w.q_len, w.H, w.causal)
        mla.decode_streaming(q8, sq, qr[b].reshape(-1, 64), c8, sk, kr, w.tau, vis)
        el += time.perf_counter() - ts
        toks += N
        seqs += 1
        if el > budget_s and seqs >= 2:
            break
    res = {"value": round(toks * BYTES_PER_TOKEN / el / 1e9, 3), "unit": "GB/s", "cores": threads,
           "kind": "oracle",
           "sample": f"{seqs} of {w.B} sequences ({toks} KV tokens, {w.H * w.q_len} rows each): per-token "
                     f"quantization + decode_streaming in float64, {el:.1f} s; the full step extrapolates to "
                     f"{el * w.total_tokens / toks:.1f} s"}
    # the same oracle with one BLAS thread, on the first sequence
    try:
        from threadpoolctl import threadpool_limits
        N = int(w.seq_lens[0])
        ck, kr = w.tokens(0, 0, N)
        with threadpool_limits(limits=1):
            ts = time.perf_counter()
            q8, sq = quant.quantize_rows(qn[0].reshape(-1, 512))
            c8, sk = quant.quantize_rows(ck)
            mla.decode_streaming(q8, sq, qr[0].reshape(-1, 64), c8, sk, kr, w.tau,
                                 mla.visible_counts(N, w.q_len, w.H, w.causal))
            el1 = time.perf_counter() - ts
        res["one_thread"] = {"value": round(N * BYTES_PER_TOKEN / el1 / 1e9, 4), "unit": "GB/s",
                             "sample": f"sequence 0 ({N} KV tokens), {el1:.1f} s"}
    except Exception:  # pragma: no cover
        pass
    return res


FETCH_BYTES_PER_TOKEN = BYTES_PER_TOKEN + 2 * (512 + 64)     # cache row read + bf16 row written


def fetch_cpu_baseline(w, run, budget_s=10.0):
    """The oracle's fetch_dequant, as written, on whole sequences of the device cache until ~budget_s."""
    import torch
    from oracle import fetch
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = 1
    el, toks, seqs = 0.0, 0, 0
    for b in range(w.B):
        n = int(w.seq_lens[b])
        npg = (n + 63) // 64
        pages = run.page_table[b, :npg].long()
        lat = run.kv_latent[pages].cpu().numpy()
        sc = run.kv_scale[pages].cpu().numpy()
        rope = run.k_rope[pages].view(torch.int16).cpu().numpy().view("uint16")
        import numpy as np
        pt = np.arange(npg, dtype=np.int32)[None]
        ts = time.perf_counter()
        fetch.fetch_dequant(lat, sc, rope, pt, np.array([0, n]))
        el += time.perf_counter() - ts
        toks += n
        seqs += 1
        if el > budget_s and seqs >= 2:
            break
    return {"value": round(toks * FETCH_BYTES_PER_TOKEN / el / 1e9, 3), "unit": "GB/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{seqs} of {w.B} sequences ({toks} tokens): oracle fetch_dequant over pages read back from "
                      f"the device cache, {el:.1f} s"}


def bench_fetch(args, w, run):
    """snapmla_fetch_dequant over every cached token of the workload (one launch per call)."""
    import numpy as np
    import torch
    from paper_2602_10718_amd import snapmla as sm
    run.append()                       # the step's tokens too: every counted token is in the cache
    torch.cuda.synchronize()
    cu = np.concatenate([[0], np.cumsum(w.seq_lens)]).astype(np.int32)
    cu_d = torch.from_numpy(cu).cuda()
    out = torch.empty((int(cu[-1]), 576), dtype=torch.bfloat16, device="cuda")
    stream = torch.cuda.current_stream()

    def call():
        sm.snapmla_fetch_dequant(run.kv_latent, run.kv_scale, run.k_rope, run.page_table, cu_d, out)

    if args.traffic_probe:
        src = torch.ones(1 << 26, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        for _ in range(3):
            call()
            torch.cuda.synchronize()
        print(json.dumps({"traffic_probe": True, "op": "fetch_dequant", "copy_bytes_read": src.numel() * 4,
                          "calls": 3, "tokens": int(cu[-1])}), flush=True)
        return

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(args.steps):
        call()
    b.record(stream)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / args.steps
    nbytes = int(cu[-1]) * FETCH_BYTES_PER_TOKEN
    gbps = nbytes / (ms * 1e-3) / 1e9
    _log(f"fetch_dequant: {ms * 1e3:.1f} us/call, {gbps:.0f} GB/s")
    # context: a plain device copy moving the same number of bytes (half read, half written)
    src = torch.empty(nbytes // 2 // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    a.record(stream)
    for _ in range(10):
        dst.copy_(src)
    b.record(stream)
    torch.cuda.synchronize()
    copy_ms = a.elapsed_time(b) / 10
    del src, dst
    copy_ref = {"bytes": nbytes // 2 // 4 * 4 * 2, "us": round(copy_ms * 1e3, 1),
                "GBps": round(nbytes / (copy_ms * 1e-3) / 1e9, 1)}
    _log(f"device copy of the same bytes: {copy_ref}")
    line = {
        "metric": "fetch-dequant GB/s (644 B read + 1152 B written per cached token)",
        "value": round(gbps, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4), "us_per_step": round(ms * 1e3, 1), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "e4m3->bf16", "data": "synthetic",
        "config": {"workload": wl_describe(args.workload) + " cache, every token fetched", "tokens": int(cu[-1]),
                   "sequences": w.B, "bytes_per_call": nbytes, "step": "snapmla_fetch_dequant"},
        "roofline": {"bound": "hbm", "kernel": "fetch_dequant_kernel, HIP events on its stream",
                     "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(gbps / HBM_PEAK_GBPS, 4), "traffic": _traffic("fetch_" + w.name, "fetch_dequant"),
                     "algorithmic_bytes_per_launch": nbytes},
        "device_copy_same_bytes": copy_ref,
    }
    if not args.no_cpu_baseline:
        _log("cpu baseline (oracle) ...")
        line["cpu_baseline"] = fetch_cpu_baseline(w, run)
    print(json.dumps(line), flush=True)


BF16_BYTES_PER_TOKEN = 2 * 512 + 2 * 64     # bf16 latent + bf16 rope


def bf16_cpu_baseline(w, budget_s=15.0):
    """The oracle's float64 attention on the bf16 inputs (mla.bf16_reference), on a bounded sample."""
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = 1
    from oracle import mla
    qn, qr = w.queries()
    el, toks, seqs = 0.0, 0, 0
    for b in range(w.B):
        N = int(w.seq_lens[b])
        ck, kr = w.tokens(b, 0, N)
        ts = time.perf_counter()
        mla.bf16_reference(qn[b].reshape(-1, 512), qr[b].reshape(-1, 64), ck, kr, w.tau,
                           mla.visible_counts(N, w.q_len, w.H, w.causal))
        el += time.perf_counter() - ts
        toks += N
        seqs += 1
        if el > budget_s and seqs >= 2:
            break
    return {"value": round(toks * BF16_BYTES_PER_TOKEN / el / 1e9, 3), "unit": "GB/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{seqs} of {w.B} sequences ({toks} KV tokens, {w.H * w.q_len} rows each): bf16_reference "
                      f"in float64, {el:.1f} s"}


def bench_bf16(args, w, run8):
    """The BF16-cache step (append_bf16 + decode_bf16 + combine) on the same workload, timed beside the
    FP8 step: the paper's FP8-vs-BF16 decode comparison on one MI355X."""
    import numpy as np
    import torch
    from paper_2602_10718_amd.runner import DecodeRunner
    t0 = time.perf_counter()
    run16 = DecodeRunner(w, num_splits=run8.num_splits, out_dtype=torch.bfloat16, kv_dtype="bf16")
    _log(f"bf16 cache filled in {time.perf_counter() - t0:.1f} s")
    stream = torch.cuda.current_stream()

    if args.traffic_probe:
        src = torch.ones(1 << 26, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        for _ in range(3):
            run16.decode()
            torch.cuda.synchronize()
        print(json.dumps({"traffic_probe": True, "op": "decode_bf16", "copy_bytes_read": src.numel() * 4,
                          "decode_calls": 3, "workload": w.name}), flush=True)
        return

    def timed(fn, k):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(k):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / k * 1e3

    def per_call(run):
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
        for k in range(args.steps):
            run.append()
            ev[k][0].record(stream)
            run.decode()
            ev[k][1].record(stream)
            run.combine()
            ev[k][2].record(stream)
        torch.cuda.synchronize()
        return (float(np.mean([e[0].elapsed_time(e[1]) for e in ev])) * 1e3,
                float(np.mean([e[1].elapsed_time(e[2]) for e in ev])) * 1e3)

    # both legs as three calls (append, decode, combine), so that the two steps have the same
    # launch structure (the FP8 path's fused snapmla_append_decode has no BF16 counterpart)
    def split_step(run):
        return lambda: (run.append(), run.decode(), run.combine())

    res = {}
    for name, run in (("fp8", run8), ("bf16", run16)):
        for _ in range(args.warmup):
            split_step(run)()
        step_us = timed(split_step(run), args.steps)
        dec_us, comb_us = per_call(run)
        res[name] = {"step_us": round(step_us, 1), "decode_us": round(dec_us, 1), "combine_us": round(comb_us, 1)}
        _log(f"{name}: step {step_us:.1f} us, decode {dec_us:.1f} us, combine {comb_us:.1f} us")
    # interleaved repeat, so that a clock drift between the two legs does not decide the ratio
    f8b = [timed(split_step(run8), args.steps) for _ in range(3)]
    b16b = [timed(split_step(run16), args.steps) for _ in range(3)]
    kv16 = w.total_tokens * BF16_BYTES_PER_TOKEN
    kv8 = w.kv_bytes()
    us16 = res["bf16"]["step_us"]
    dec16 = res["bf16"]["decode_us"]
    flops = 2.0 * w.total_tokens * 64 * ((w.H * w.q_len + 63) // 64) * (576 + 512)
    gbps = kv16 / (us16 * 1e-6) / 1e9
    dec_gbps = kv16 / (dec16 * 1e-6) / 1e9
    line = {
        "metric": "BF16-cache MLA decode µs/step + KV HBM GB/s beside the FP8 step, 64 heads, 8K-32K ctx",
        "value": round(gbps, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(us16 * 1e-3, 4), "us_per_step": us16, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl_describe(args.workload) + ", BF16 cache (1152 B per token)", "batch": w.B,
                   "heads": w.H, "q_len": w.q_len, "kv_tokens": w.total_tokens, "kv_bytes_bf16": kv16,
                   "kv_bytes_fp8": kv8, "num_splits": run16.num_splits,
                   "step": "append_bf16 + decode_bf16 + combine (FP8 leg: quantize_append + decode + combine), three calls each"},
        "fp8": res["fp8"], "bf16": res["bf16"],
        "speedup_fp8_over_bf16": {"step": round(us16 / res["fp8"]["step_us"], 3),
                                  "decode_call": round(dec16 / res["fp8"]["decode_us"], 3),
                                  "step_repeats": [round(b / a, 3) for a, b in zip(f8b, b16b)],
                                  "kv_byte_ratio": round(kv16 / kv8, 3)},
        "roofline": {"bound": "hbm", "kernel": "snapmla_decode_bf16 call (prep_kernel + decode_bf16_kernel), "
                                               "HIP events on its stream",
                     "achieved": round(dec_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(dec_gbps / HBM_PEAK_GBPS, 4), "traffic": _traffic("bf16_" + w.name, "decode_bf16"),
                     "algorithmic_bytes_per_launch": kv16,
                     "mfma_frac_bf16": round(flops / (dec16 * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 4)},
    }
    if not args.no_cpu_baseline:
        _log("cpu baseline (oracle bf16_reference) ...")
        line["cpu_baseline"] = bf16_cpu_baseline(w)
    print(json.dumps(line), flush=True)


FP8_PEAK_TFLOPS = 5000.0       # dense FP8 MFMA
BF16_PEAK_TFLOPS = 2500.0      # dense BF16 MFMA


def bench_sweep(args):
    """Decode + combine of the same batch-32 cache for every (H, q_len) of the sweep."""
    import numpy as np
    import torch
    from paper_2602_10718_amd import workloads as wl
    from paper_2602_10718_amd.runner import DecodeRunner
    stream = torch.cuda.current_stream()
    base = None
    rows = []
    t_fill = time.perf_counter()

    def timed(fn, k):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(k):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / k * 1e3

    for q_len in wl.SWEEP_QLEN:
        for H in wl.SWEEP_HEADS:
            w = wl.sweep(H, q_len)
            run = DecodeRunner(w, out_dtype=torch.bfloat16,
                               cache=None if base is None else (base.kv_latent, base.kv_scale, base.k_rope))
            if base is None:
                base = run
                t_fill = time.perf_counter() - t_fill
                _log(f"sweep cache filled ({w.total_tokens} tokens) in {t_fill:.1f} s")
            run.append()
            for _ in range(args.warmup):
                run.decode()
                run.combine()
            us_dec = timed(run.decode, args.steps)
            us_cmb = timed(run.combine, args.steps)
            R = H * q_len
            toks = w.total_tokens
            t_hbm = w.kv_bytes() / (HBM_PEAK_GBPS * 1e9) * 1e6
            t_mfma = toks * R * (2 * 512 * 2 / (FP8_PEAK_TFLOPS * 1e12) + 2 * 64 / (BF16_PEAK_TFLOPS * 1e12)) * 1e6
            e = {"H": H, "q_len": q_len, "rows": R, "causal": bool(w.causal), "num_splits": run.num_splits,
                 "decode_us": round(us_dec, 1), "combine_us": round(us_cmb, 1),
                 "kv_GBps": round(w.kv_bytes() / (us_dec * 1e-6) / 1e9, 1),
                 "hbm_roofline_us": round(t_hbm, 1), "mfma_roofline_us": round(t_mfma, 1),
                 "bound": "mfma" if t_mfma > t_hbm else "hbm",
                 "frac_hbm": round(t_hbm / us_dec, 4), "frac_mfma": round(t_mfma / us_dec, 4)}
            e["frac"] = max(e["frac_hbm"], e["frac_mfma"])
            rows.append(e)
            _log(f"H={H} q_len={q_len}: decode {us_dec:.1f} us ({e['kv_GBps']} GB/s, {e['bound']} frac {e['frac']})")
            del run
    w = wl.sweep(64, 1)
    line = {"metric": "sensitivity sweep: snapmla_decode us and roofline fraction per (H, q_len)",
            "unit": "us", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "higher_is_better": False,
            "dtype": "e4m3", "data": "synthetic",
            "config": {"workload": "batch 32, lengths U[16384, 131072], shared cache", "batch": w.B,
                       "kv_tokens": w.total_tokens, "kv_bytes": w.kv_bytes(), "heads": list(wl.SWEEP_HEADS),
                       "q_len": list(wl.SWEEP_QLEN), "peaks": {"hbm_GBps": HBM_PEAK_GBPS,
                                                               "fp8_TFLOPs": FP8_PEAK_TFLOPS,
                                                               "bf16_TFLOPs": BF16_PEAK_TFLOPS}},
            "sweep": rows}
    print(json.dumps(line), flush=True)


def torch_attention_f32(qn, qr, ckv, kr, tau, visible):
    """fp32 softmax attention on bf16 inputs (device tensors, bfloat16): the unquantized reference the
    ablation scores against.  s = tau (q_nope c^T + q_rope k_r^T); o = softmax(s) c; row r sees the
    first visible[r] tokens.  Returns float32 [R, 512]."""
    import torch
    q1, q2 = qn.float(), qr.float()
    c, k = ckv.float(), kr.float()
    s = tau * (q1 @ c.t().contiguous() + q2 @ k.t().contiguous())
    N = c.shape[0]
    mask = torch.arange(N, device=s.device)[None, :] >= torch.as_tensor(visible, device=s.device)[:, None]
    s = s.masked_fill(mask, float("-inf"))
    return torch.softmax(s, dim=1) @ c


def bench_ablation(args):
    """Each cache granularity of the accuracy ablation: quantizer time, decode error vs fp32 attention."""
    import numpy as np
    import torch
    from paper_2602_10718_amd import snapmla as sm
    from paper_2602_10718_amd import workloads as wl
    from paper_2602_10718_amd.runner import DecodeRunner
    w = wl.ablation(B=32, H=16, ctx=8192)
    stream = torch.cuda.current_stream()
    run = DecodeRunner(w, out_dtype=torch.float32, fill=False)
    T = w.total_tokens
    ck = np.empty((T, 512), np.uint16)
    kr = np.empty((T, 64), np.uint16)
    cu = np.concatenate([[0], np.cumsum(w.seq_lens)]).astype(np.int32)
    for b in range(w.B):
        ck[cu[b]:cu[b + 1]], kr[cu[b]:cu[b + 1]] = w.tokens(b, 0, int(w.seq_lens[b]))
    ck_d = torch.from_numpy(ck.view(np.int16)).cuda().view(torch.bfloat16)
    kr_d = torch.from_numpy(kr.view(np.int16)).cuda().view(torch.bfloat16)
    cu_d = torch.from_numpy(cu).cuda()
    scratch = torch.zeros(4, dtype=torch.int32, device="cuda")
    # the reference, once: fp32 attention on the bf16 inputs, row by row of every sequence
    refs = []
    for b in range(w.B):
        vis = np.full(w.H, int(w.seq_lens[b]))
        refs.append(torch_attention_f32(run.q_nope[b].reshape(-1, 512), run.q_rope[b].reshape(-1, 64),
                                        ck_d[cu[b]:cu[b + 1]], kr_d[cu[b]:cu[b + 1]], w.tau, vis))
    ref = torch.cat(refs).double()
    rows = []
    qbytes = T * (2 * (512 + 64) + 512 + 4 + 2 * 64)       # bf16 rows read, cache planes written
    for name in ("snapmla", "A", "B", "C", "D"):
        def quant():
            sm.snapmla_quantize_cache_config(ck_d, kr_d, run.page_table, cu_d, name, run.kv_latent, run.kv_scale,
                                             run.k_rope, scratch=scratch)
        for _ in range(args.warmup):
            quant()
        torch.cuda.synchronize()
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(args.steps):
            quant()
        e.record(stream)
        torch.cuda.synchronize()
        us = a.elapsed_time(e) / args.steps * 1e3
        run.decode()
        run.combine()
        torch.cuda.synchronize()
        o = run.out.reshape(-1, 512).double()
        d = o - ref
        cos = torch.sum(o * ref, dim=1) / (torch.linalg.norm(o, dim=1) * torch.linalg.norm(ref, dim=1))
        r = {"config": name, "quantize_us": round(us, 1), "quantize_GBps": round(qbytes / (us * 1e-6) / 1e9, 1),
             "rmse": float(torch.sqrt(torch.mean(d * d))), "cos_diff": float(torch.mean(1 - cos)),
             "rel_l2": float(torch.linalg.norm(d) / torch.linalg.norm(ref))}
        rows.append(r)
        _log(f"{name}: quantize {us:.1f} us, rel_l2 {r['rel_l2']:.3e}, 1-cos {r['cos_diff']:.3e}, rmse {r['rmse']:.3e}")
    line = {"metric": "KV-cache quantization granularity ablation: decode error vs fp32 attention on bf16 inputs",
            "unit": "rel_l2", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "higher_is_better": False,
            "dtype": "e4m3", "data": "synthetic",
            "config": {"workload": "ablation: B32 H16 ctx8192, content ~1e0-1e1 (x20 outliers), RoPE ~1e3",
                       "tokens": T, "quantize_bytes_per_call": qbytes,
                       "configs": {"snapmla": "per-token RoPE-aware", "A": "per-token RoPE-unaware",
                                   "B": "per-tensor static 1.0", "C": "per-tensor dynamic", "D": "per-block"}},
            "ablation": rows}
    print(json.dumps(line), flush=True)


def read_ceiling(run, w, timed, units=256, reps=50):
    """Time snapmla_debug_read_ceiling over the decode's pages: every 64-token block of every
    sequence in order, streamed into LDS with the decode's copy structure and no attention
    arithmetic, one workgroup per CU as in the decode launch.  Returns its time, its rate in
    bytes of whole pages (41,216 B per block), and the ceiling's time over the decode call's
    (decode_call_frac, filled in by the caller)."""
    import numpy as np
    import torch
    from paper_2602_10718_amd import snapmla as sm
    npg = (w.seq_lens.astype(np.int64) + 63) // 64
    pages = np.concatenate([w.page_table[b, :npg[b]] for b in range(w.B)]).astype(np.int32)
    pages_d = torch.from_numpy(pages).cuda()
    units = max(units, -(-len(pages) // 1792))
    out = torch.empty(units, dtype=torch.int32, device="cuda")

    def call():
        sm.snapmla_debug_read_ceiling(run.kv_latent, run.kv_scale, run.k_rope, pages_d, run.kv_latent.shape[0],
                                      units, out)
    for _ in range(20):
        call()
    ms = timed(call, reps)
    page_bytes = len(pages) * 41216
    return {"kernel": "read_ceiling_kernel (snapmla_debug_read_ceiling), HIP events", "units": units,
            "blocks": len(pages), "us": round(ms * 1e3, 1), "page_bytes": page_bytes,
            "GBps": round(page_bytes / (ms * 1e-3) / 1e9, 1)}


def plain_stream(nbytes, timed, grid=2048, reps=20):
    """Time snapmla_debug_read_stream over a buffer of `nbytes` (the KV bytes of the workload): the
    plain 16-byte-load read stream, the memory system's rate for the simplest streaming kernel."""
    import torch
    from paper_2602_10718_amd import snapmla as sm
    n = (nbytes + 15) // 16 * 16
    buf = torch.ones(n // 4, dtype=torch.int32, device="cuda")
    out = torch.empty(grid, dtype=torch.int32, device="cuda")

    def call():
        sm.snapmla_debug_read_stream(buf, grid, out)
    for _ in range(5):
        call()
    ms = timed(call, reps)
    del buf
    return {"kernel": "read_stream_kernel (snapmla_debug_read_stream), HIP events", "grid": grid, "bytes": n,
            "us": round(ms * 1e3, 1), "GBps": round(n / (ms * 1e-3) / 1e9, 1)}


def accuracy_vs_bf16(run, w, samples=8):
    """Error of the step's output against an unquantized reference: fp32 softmax attention on the same
    bf16 inputs (plain torch on the GPU), over `samples` sequences spread over the batch.  The decode is
    merged into a float32 output so that the figure is the kernel's, not the output rounding's."""
    import numpy as np
    import torch
    from paper_2602_10718_amd import snapmla as sm
    out32 = torch.empty((w.B, w.q_len, w.H, 512), dtype=torch.float32, device="cuda")
    lse32 = torch.empty((w.B, w.q_len, w.H), dtype=torch.float32, device="cuda")
    # (the decode writes the rows it finalises itself into the same float32 output)
    sm.snapmla_append_decode(run.new_ckv, run.new_krope, run.q_nope, run.q_rope, run.kv_latent, run.kv_scale,
                             run.k_rope, run.page_table, run.seq_lens, w.tau, w.causal, run.num_splits,
                             run.kv_chunk_tokens, run.workspace, flags=run.flags, out=out32, lse=lse32)
    sm.snapmla_combine(run.workspace, run.seq_lens, w.B, w.q_len, w.H, run.num_splits, run.kv_chunk_tokens, out32,
                       lse32)
    torch.cuda.synchronize()
    picks = sorted(set(np.linspace(0, w.B - 1, min(samples, w.B)).round().astype(int).tolist()))
    num = den = sse = 0.0
    cos_sum, rows, worst = 0.0, 0, 0.0
    for b in picks:
        N = int(w.seq_lens[b])
        if N == 0:
            continue
        ck, kr = w.tokens(b, 0, N)
        c = torch.from_numpy(ck.view(np.int16)).cuda().view(torch.bfloat16)
        k = torch.from_numpy(kr.view(np.int16)).cuda().view(torch.bfloat16)
        vis = [N - w.q_len + 1 + t if w.causal else N for t in range(w.q_len) for _ in range(w.H)]
        ref = torch_attention_f32(run.q_nope[b].reshape(-1, 512), run.q_rope[b].reshape(-1, 64), c, k, w.tau,
                                  vis).double()
        o = out32[b].reshape(-1, 512).double()
        d = o - ref
        num += float(torch.sum(d * d))
        den += float(torch.sum(ref * ref))
        cos = torch.sum(o * ref, dim=1) / (torch.linalg.norm(o, dim=1) * torch.linalg.norm(ref, dim=1))
        cos_sum += float(torch.sum(1 - cos))
        rows += o.shape[0]
        worst = max(worst, float(torch.max(torch.max(torch.abs(d), dim=1).values
                                           / torch.clamp(torch.max(torch.abs(ref), dim=1).values, min=1.0))))
    return {"reference": "fp32 softmax attention on the bf16 inputs (torch on the GPU), float32 merge output",
            "sequences": picks, "rows": rows, "rel_l2": float(np.sqrt(num / den)),
            "rmse": float(np.sqrt(num / (rows * 512))), "one_minus_cos": cos_sum / rows,
            "max_abs_over_row_scale": worst}


def wl_describe(name):
    from paper_2602_10718_amd import workloads as wl
    return wl.describe(name)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=1000)
    ap.add_argument("--workload", default="headline",
                    choices=("tiny", "dsv3", "headline", "longsplit", "mtp"), help="workload by name")
    ap.add_argument("--num-splits", type=int, default=None)
    ap.add_argument("--plan", default="auto", choices=["auto", "balanced", "unsplit"],
                    help="split plan: balanced block ranges (+ combine), one piece per sequence (no combine), or "
                         "auto: the unsplit plan where the runner expects it to be faster (small batches)")
    ap.add_argument("--cold-steps", type=int, default=50, help="cold-cache steps (0 to skip)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--op", default="decode", choices=["decode", "fetch_dequant", "sweep", "ablation", "decode_bf16"],
                    help="decode: the hot path step (default); fetch_dequant: snapmla_fetch_dequant over every "
                         "cached token of the workload; sweep: decode + combine for H in 16..128 x q_len in {1, 2} "
                         "at batch 32, lengths U[16K, 128K]; ablation: the cache quantized under each granularity "
                         "of the accuracy ablation, decode error vs fp32 attention on the bf16 inputs; decode_bf16: the "
                         "BF16-cache step on the same workload, timed beside the FP8 step")
    ap.add_argument("--traffic-probe", action="store_true",
                    help="for rocprofv3 --pmc runs: one 256 MiB device copy (counter calibration), then 3 "
                         "snapmla_decode calls; prints what it ran and exits")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the decode path shards by "
              "sequence / head / KV chunk without collectives)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2602_10718_amd import workloads as wl
    from paper_2602_10718_amd.runner import DecodeRunner

    torch.cuda.set_device(0)
    if args.op == "sweep":
        bench_sweep(args)
        return
    if args.op == "ablation":
        bench_ablation(args)
        return
    w = wl.make(args.workload)
    t_fill = time.perf_counter()
    run = DecodeRunner(w, num_splits=args.num_splits, out_dtype=torch.bfloat16,
                       unsplit={"auto": "auto", "balanced": False, "unsplit": True}[args.plan])
    t_fill = time.perf_counter() - t_fill
    _log(f"cache filled ({w.total_tokens} tokens) in {t_fill:.1f} s")
    stream = torch.cuda.current_stream()
    kv_bytes = w.kv_bytes()

    if args.op == "fetch_dequant":
        bench_fetch(args, w, run)
        return
    if args.op == "decode_bf16":
        bench_bf16(args, w, run)
        return

    if args.traffic_probe:
        src = torch.ones(1 << 26, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        for _ in range(3):
            run.decode()
            torch.cuda.synchronize()
        print(json.dumps({"traffic_probe": True, "copy_bytes_read": src.numel() * 4,
                          "copy_bytes_written": dst.numel() * 4, "decode_calls": 3, "workload": w.name,
                          "kv_bytes": kv_bytes}), flush=True)
        return

    def timed(fn, k):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(k):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / k

    # ---- warm-up, then the timed region: K back-to-back steps ---------------
    # (the warm-up is long enough, ~0.2 s at the default, for the GPU's clocks to
    # settle under this load: after 20 steps the first timed steps still ran ~9 %
    # slower than after 1,000)
    for _ in range(args.warmup):
        run.step()
    torch.cuda.synchronize()
    ms_per_step = timed(run.step, args.steps)
    _log(f"timed {args.steps} steps: {ms_per_step * 1e3:.1f} us/step")

    # ---- the same step as a HIP graph replay --------------------------------
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run.step()
    for _ in range(20):
        graph.replay()
    graph_us = timed(graph.replay, args.steps) * 1e3
    _log(f"graph replay: {graph_us:.1f} us/step")

    # ---- the same step issued eagerly, with the per-call split ---------------
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for k in range(args.steps):
        ev[k][0].record(stream)
        run.append()
        ev[k][1].record(stream)
        run.decode()
        ev[k][2].record(stream)
        if run.needs_combine:
            run.combine()
        ev[k][3].record(stream)
    torch.cuda.synchronize()
    step_each = np.array([e[0].elapsed_time(e[3]) for e in ev]) * 1e3
    append_us = float(np.mean([e[0].elapsed_time(e[1]) for e in ev])) * 1e3
    decode_us = float(np.mean([e[1].elapsed_time(e[2]) for e in ev])) * 1e3
    combine_us = float(np.mean([e[2].elapsed_time(e[3]) for e in ev])) * 1e3
    _log(f"per call: append {append_us:.1f} decode {decode_us:.1f} combine {combine_us:.1f} us")

    # ---- the decode kernel alone: the decode launch without its preparation launch,
    # over the workspace the calls above prepared (the dominant kernel of the roofline)
    kernel_us = timed(run.decode_kernel_only, args.steps) * 1e3
    _log(f"decode kernel alone: {kernel_us:.1f} us")

    # ---- cold cache: 1 GiB scratch write + read between steps (not timed) ----
    cold = None
    if args.cold_steps > 0:
        scratch = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        sink = torch.empty((), dtype=torch.float32, device="cuda")
        ts = []
        for k in range(args.cold_steps):
            scratch.fill_(float(k))
            sink.copy_(scratch.sum())
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            run.step()
            b.record(stream)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b) * 1e3)
        del scratch, sink
        cold = {"steps": args.cold_steps, "median_us": round(float(np.median(ts)), 1),
                "p90_us": round(float(np.percentile(ts, 90)), 1),
                "median_GBps": round(kv_bytes / (float(np.median(ts)) * 1e-6) / 1e9, 1)}
        _log(f"cold: median {cold['median_us']} us, p90 {cold['p90_us']} us")

    # ---- the exact-accumulation QK mode, same cache, same plan ----------------
    run_x = DecodeRunner(w, num_splits=run.num_splits, kv_chunk_tokens=run.kv_chunk_tokens, out_dtype=torch.bfloat16,
                         cache=(run.kv_latent, run.kv_scale, run.k_rope), exact_qk=True)
    for _ in range(args.warmup):
        run_x.step()
    torch.cuda.synchronize()
    exact_ms = timed(run_x.step, args.steps)
    exact_dec_us = timed(run_x.append_decode, args.steps) * 1e3
    _log(f"exact-QK mode: {exact_ms * 1e3:.1f} us/step, append_decode {exact_dec_us:.1f} us")

    # ---- read-stream ceiling over the same pages (a measurement kernel) --------
    ceiling = read_ceiling(run, w, timed)
    _log(f"read-stream ceiling: {ceiling['us']} us, {ceiling['GBps']} GB/s of whole pages")
    stream_ref = plain_stream(kv_bytes, timed)
    _log(f"plain read stream: {stream_ref['us']} us, {stream_ref['GBps']} GB/s")

    # ---- error against the unquantized (bf16-input, fp32) reference -----------
    acc = {"fp8_qk": accuracy_vs_bf16(run, w), "exact_qk": accuracy_vs_bf16(run_x, w)}
    _log(f"vs bf16 reference: rel_l2 {acc['fp8_qk']['rel_l2']:.3e} (FP8 QK), {acc['exact_qk']['rel_l2']:.3e} (exact QK)")
    del run_x

    gbps = kv_bytes / (ms_per_step * 1e-3) / 1e9
    decode_gbps = kv_bytes / (decode_us * 1e-6) / 1e9
    kernel_gbps = kv_bytes / (kernel_us * 1e-6) / 1e9
    ceiling["decode_call_frac"] = round(ceiling["us"] / decode_us, 4)
    ceiling["decode_kernel_frac"] = round(ceiling["us"] / kernel_us, 4)
    traffic = _traffic(w.name, "decode", kernel="decode_kernel")
    # the bound of the decode call: KV bytes at 8 TB/s against its MFMA work at the dense
    # peaks (2 x 512 FP8 QK + 2 x 512 FP8 PV + 2 x 64 BF16 RoPE FLOP per token and row)
    R = w.H * w.q_len
    t_hbm = kv_bytes / (HBM_PEAK_GBPS * 1e9) * 1e6
    t_mfma = w.total_tokens * R * (2 * 512 * 2 / (FP8_PEAK_TFLOPS * 1e12) + 2 * 64 / (BF16_PEAK_TFLOPS * 1e12)) * 1e6
    kern = ("decode_kernel alone (snapmla_debug_decode_kernel over the workspace a snapmla_decode call prepared), "
            "HIP events on its stream")
    call = {"what": "the whole snapmla_decode call (prep_kernel + decode_kernel), HIP events on its stream",
            "us": round(decode_us, 2), "traffic": _traffic(w.name, "decode")}
    if t_mfma > t_hbm:
        fp8_eq = w.total_tokens * R * (2 * 512 * 2 + 2 * 64 * 2)      # BF16 FLOPs count twice at the FP8 rate
        achieved = fp8_eq / (kernel_us * 1e-6) / 1e12
        call_achieved = fp8_eq / (decode_us * 1e-6) / 1e12
        call.update(achieved=round(call_achieved, 1), frac=round(call_achieved / FP8_PEAK_TFLOPS, 4))
        roofline = {"bound": "mfma", "kernel": kern, "kernel_us": round(kernel_us, 2), "achieved": round(achieved, 1),
                    "peak": FP8_PEAK_TFLOPS, "unit": "TFLOP/s (FP8-equivalent: BF16 FLOPs counted twice)",
                    "frac": round(achieved / FP8_PEAK_TFLOPS, 4), "traffic": traffic,
                    "algorithmic_flops_per_launch": fp8_eq, "hbm_frac": round(kernel_gbps / HBM_PEAK_GBPS, 4)}
    else:
        call.update(achieved=round(decode_gbps, 1), frac=round(decode_gbps / HBM_PEAK_GBPS, 4))
        roofline = {"bound": "hbm", "kernel": kern, "kernel_us": round(kernel_us, 2), "achieved": round(kernel_gbps, 1),
                    "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(kernel_gbps / HBM_PEAK_GBPS, 4),
                    "traffic": traffic, "algorithmic_bytes_per_launch": kv_bytes}
    roofline["decode_call"] = call
    roofline["read_ceiling"] = ceiling
    stream_ref["decode_call_frac"] = round(stream_ref["us"] / decode_us, 4)
    stream_ref["decode_kernel_frac"] = round(stream_ref["us"] / kernel_us, 4)
    roofline["plain_stream"] = stream_ref
    line = {
        "metric": METRIC,
        "value": round(gbps, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "us_per_step": round(ms_per_step * 1e3, 1),
        "frac_of_hbm_peak": round(gbps / HBM_PEAK_GBPS, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "e4m3",
        "data": "synthetic",
        "config": {
            "workload": wl.describe(args.workload),
            "batch": w.B, "heads": w.H, "q_len": w.q_len, "causal": bool(w.causal),
            "ctx_min": int(w.seq_lens.min()), "ctx_max": int(w.seq_lens.max()),
            "kv_tokens": w.total_tokens, "kv_bytes": kv_bytes, "page": 64,
            "num_splits": run.num_splits, "kv_chunk_tokens": run.kv_chunk_tokens,
            "append_per_step": w.n_new,
            "step": "append + decode + combine" if run.needs_combine else "append + decode (unsplit plan, rows written by the decode)",
        },
        "us_per_step_graph": round(graph_us, 1),
        "breakdown_us": {"append": round(append_us, 2), "decode": round(decode_us, 2),
                         "combine": round(combine_us, 2)},
        "warm_step_us_each": {"steps": args.steps, "median": round(float(np.median(step_each)), 1),
                              "p90": round(float(np.percentile(step_each, 90)), 1)},
        "cold_cache": cold,
        "qk_mode": "FP8 matrix cores (flags 0)",
        "exact_qk": {"flags": "SNAPMLA_DECODE_EXACT_QK", "us_per_step": round(exact_ms * 1e3, 1),
                     "GBps": round(kv_bytes / (exact_ms * 1e-3) / 1e9, 1),
                     "append_decode_us": round(exact_dec_us, 1)},
        "accuracy_vs_bf16": acc,
        "roofline": roofline,
        "cache_fill_s": round(t_fill, 1),
    }
    if not args.no_cpu_baseline:
        _log("cpu baseline (oracle) ...")
        line["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
