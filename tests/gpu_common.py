"""Shared helpers of the GPU parity tests: run the HIP path, compute the oracle, compare."""

import numpy as np
import torch

from oracle import check
from paper_2602_10718_amd import workloads as wl_mod


def runner(wl, **kw):
    from paper_2602_10718_amd.runner import DecodeRunner
    return DecodeRunner(wl, **kw)


def qk_mode(run):
    """The oracle's QK mode matching a runner's decode flags."""
    return "exact" if run.flags & 1 else "mfma8"


def reference(wl, b, qn=None, qr=None, qk="mfma8"):
    """Oracle results for sequence b of workload wl (regenerated from the seeds), with the content
    term formed as the decode forms it: "mfma8" for the default decode (FP8 matrix cores), "exact"
    for a runner made with exact_qk=True."""
    if qn is None:
        qn, qr = wl.queries()
    N = int(wl.seq_lens[b])
    ck, kr = wl.tokens(b, 0, N)
    return check.sequence_reference(qn[b], qr[b], ck, kr, wl.tau, wl.q_len, wl.H, wl.causal, qk=qk)


def check_sequence(run, b, ref, strict_north_star=True, label=""):
    """Compare the device output/LSE of sequence b with the oracle; returns the metrics.

    Asserts the derived per-element bounds (oracle/check.bounds) and, with strict_north_star, the
    the benchmark spec tolerance (check.north_star: LSE within max(1e-3, 2^-18 |LSE|), per-row max abs
    within 2e-2 max(1, max|o_r|) plus tie slack, relative L2 within 1e-2)."""
    assert ref["qk"] == qk_mode(run), f"{label}: oracle QK mode {ref['qk']} for a {qk_mode(run)} decode"
    R = run.q_len * run.H
    o = run.out[b].reshape(R, 512).float().cpu().numpy().astype(np.float64)
    lse = run.lse[b].reshape(R).cpu().numpy().astype(np.float64)
    ob, lb, info = check.bounds(ref)
    err = np.abs(o - ref["o"])
    lerr = np.abs(lse - ref["lse"])
    fin = np.isfinite(ref["lse"])
    assert np.array_equal(np.isfinite(lse), fin), f"{label}: LSE finiteness differs"
    assert np.all(lse[~fin] == -np.inf) and np.all(o[~fin] == 0), f"{label}: rows without tokens must be 0/-inf"
    assert np.all(np.isfinite(o)), f"{label}: non-finite output"
    m = check.metrics(o, lse, ref["o"], ref["lse"])
    m_bf = check.metrics(o, lse, ref["o_bf16"], ref["lse_bf16"])
    m["vs_bf16_rel_l2"] = m_bf["rel_l2"]
    m["ties"] = info["tie_count"]
    m["bound_violations"] = int(np.sum(err > ob))
    m["lse_violations"] = int(np.sum(lerr[fin] > lb[fin]))
    row_scale = np.maximum(1.0, np.max(np.abs(ref["o"]), axis=1))
    m["max_abs_rowrel"] = float(np.max(np.max(err, axis=1) / row_scale))
    ns_ok, ns = check.north_star(o, lse, ref, info["tie_slack"])
    m["ns_lse"], m["ns_maxabs"] = ns["lse_ratio"], ns["maxabs_ratio"]
    print(f"[{label} {ref['qk']} b={b}] " + " ".join(f"{k}={v:.3g}" if isinstance(v, float) else f"{k}={v}"
                                                    for k, v in m.items()), flush=True)
    worst = np.unravel_index(np.argmax(err - ob), err.shape)
    assert m["bound_violations"] == 0, f"{label}: {m['bound_violations']} outputs outside the derived bound; " \
        f"worst at {worst}: err {err[worst]:.3g} bound {ob[worst]:.3g}"
    assert m["lse_violations"] == 0, f"{label}: LSE outside the derived bound (max err {m['lse_max_abs']:.3g})"
    if strict_north_star:
        assert ns_ok, f"{label}: outside the north_star tolerance {ns}"
    return m


def reference_bf16(wl, b, qn=None, qr=None):
    """Oracle results of the BF16-cache decode for sequence b of workload wl."""
    if qn is None:
        qn, qr = wl.queries()
    N = int(wl.seq_lens[b])
    ck, kr = wl.tokens(b, 0, N)
    return check.sequence_reference_bf16(qn[b], qr[b], ck, kr, wl.tau, wl.q_len, wl.H, wl.causal)


def check_sequence_bf16(run, b, ref, label=""):
    """Device output/LSE of sequence b of a BF16-cache run against the oracle and its bounds."""
    R = run.q_len * run.H
    o = run.out[b].reshape(R, 512).float().cpu().numpy().astype(np.float64)
    lse = run.lse[b].reshape(R).cpu().numpy().astype(np.float64)
    ob, lb = check.bounds_bf16(ref)
    fin = np.isfinite(ref["lse"])
    assert np.array_equal(np.isfinite(lse), fin), f"{label}: LSE finiteness differs"
    assert np.all(lse[~fin] == -np.inf) and np.all(o[~fin] == 0), f"{label}: rows without tokens must be 0/-inf"
    assert np.all(np.isfinite(o)), f"{label}: non-finite output"
    err = np.abs(o - ref["o"])
    m = check.metrics(o, lse, ref["o"], ref["lse"])
    m["bound_violations"] = int(np.sum(err > ob))
    m["lse_violations"] = int(np.sum(np.abs(lse - ref["lse"])[fin] > lb[fin]))
    print(f"[{label} b={b}] " + " ".join(f"{k}={v:.3g}" if isinstance(v, float) else f"{k}={v}"
                                         for k, v in m.items()), flush=True)
    worst = np.unravel_index(np.argmax(err - ob), err.shape)
    assert m["bound_violations"] == 0, f"{label}: {m['bound_violations']} outputs outside the bound; worst at " \
        f"{worst}: err {err[worst]:.3g} bound {ob[worst]:.3g}"
    assert m["lse_violations"] == 0, f"{label}: LSE outside the bound (max err {m['lse_max_abs']:.3g})"
    assert m["rel_l2"] <= 1e-2, f"{label}: rel L2 {m['rel_l2']:.3g} > 1e-2"
    return m
