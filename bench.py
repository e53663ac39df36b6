#!/usr/bin/env python3
"""Throughput of the ESTP scoring and pooling path on one MI355X.

One step = the whole path over one batch: token entropy (fused LM-head GEMM),
attention importance (two passes), fusion + pooling, length head + SJF order,
enqueued back to back on one stream, inputs resident in HBM.  Prints one JSON
line with prompt tokens/s, the roofline position of the dominant kernel
(entropy GEMM, bf16 matrix cores) and the fp64 oracle timed on the host as a
baseline.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "prompt tokens/sec scored+pooled on 1 MI355X; % bf16 MFMA peak; pooling HBM GB/s"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 matrix peak
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 vector peak (256 CUs x 4 SIMDs x 16 lanes x 2 FLOP x 2.4 GHz)
PEAK_EXP_PER_S = 256 * 4 * 16 / 4 * 2.4e9  # v_exp_f32 at a quarter of the FMA issue rate: 9.83e12 per s
PEAK_HBM_GBPS = 8000.0      # MI355X HBM3E


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def to_dev(a, torch):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(a).cuda()


def cpu_baseline(inp, lam1, lam2, alpha, norm, n_prompts: int):
    """The fp64 oracle on a bounded sample of the same workload: its first `n_prompts`
    whole prompts through the whole path (entropy, importance, fusion, pooling, head)."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max((d.get("num_threads", 1) for d in threadpool_info()), default=1)
    except Exception:  # pragma: no cover
        blas_threads = 1
    cu = inp["cu_seqlens"].astype(np.int64)
    n_prompts = min(n_prompts, len(cu) - 1)
    n = int(cu[n_prompts])
    cu_s = cu[: n_prompts + 1]
    t0 = time.perf_counter()
    reps = 0
    while True:  # a sample that runs in well under a second is repeated, for a stable rate
        ref = oracle.run_path(inp["X"][:n], inp["W"], inp["Q"][:, :n], inp["K"][:, :n], cu_s, lam1, lam2, alpha,
                              norm, head=(inp["W1"], inp["b1"], inp["W2"], inp["b2"], inp["centres"]))
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= 2.0:
            break
    return {
        "value": reps * n / dt,
        "unit": "tokens/s",
        "cores": int(blas_threads),
        "kind": "oracle",
        "sample": (f"the first {n_prompts} whole prompts of the workload ({n} tokens), whole path"
                   + (f", {reps} times" if reps > 1 else "") + f", {dt:.1f} s"),
        "host_cpus": len(os.sched_getaffinity(0)),
    }, ref, n_prompts


def parity_of_run(ref, n_prompts: int, got: dict) -> dict:
    """This run's own outputs on the oracle's sample (its first whole prompts) against the oracle:
    the errors the parity tests bound (|dH| <= 2e-3 nats, |dS| <= 1e-3 S, pooled relative L2
    <= 1e-3, y-hat relative 1e-3)."""
    n = len(ref["H"])
    dH = float(np.abs(got["H"][:n] - ref["H"]).max())
    dS = float((np.abs(got["S"][:n] - ref["S"]) / ref["S"]).max())
    pooled = got["pooled"][:n_prompts].astype(np.float64)
    dP = float(max(np.linalg.norm(pooled[b] - ref["pooled"][b]) / np.linalg.norm(ref["pooled"][b])
                   for b in range(n_prompts)))
    dY = float((np.abs(got["yhat"][:n_prompts] - ref["yhat"]) / np.maximum(np.abs(ref["yhat"]), 1e-30)).max())
    return {"sample": f"first {n_prompts} prompts ({n} tokens)", "max_abs_dH_nats": dH, "max_rel_dS": dS,
            "max_pooled_rel_l2": dP, "max_yhat_rel": dY,
            # both sides index tokens from 0 on this sample; near ties may differ (margin rule)
            "top_token_agree": f"{int((got['top'][:n_prompts] == np.asarray(ref['top'])).sum())}/{n_prompts}",
            "within_bounds": bool(dH <= 2e-3 and dS <= 1e-3 and dP <= 1e-3 and dY <= 1e-3)}


def source_hash() -> str:
    """sha256 (16 hex digits) of the library sources, the header and this script."""
    import glob
    import hashlib
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(ROOT, "paper_2608_15592_amd", "csrc", "*")))
    files += [os.path.join(ROOT, "include", "estp.h"), os.path.abspath(__file__)]
    for f in files:
        h.update(os.path.basename(f).encode())
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def build_info(torch) -> dict:
    """Where the numbers were taken: device, runtime versions, source revision."""
    import subprocess
    props = torch.cuda.get_device_properties(0)
    rocm = None
    for f in ("/opt/rocm/.info/version", "/opt/rocm/.info/version-dev"):
        try:
            rocm = open(f).read().strip()
            break
        except OSError:
            pass
    try:
        head = subprocess.run(["git", "-C", ROOT, "rev-parse", "HEAD"], capture_output=True, text=True,
                              timeout=10).stdout.strip() or None
    except Exception:
        head = None
    return {"name": torch.cuda.get_device_name(0), "gcnArchName": getattr(props, "gcnArchName", None),
            "compute_units": props.multi_processor_count, "hbm_bytes": props.total_memory,
            "rocm": rocm, "hip_runtime": torch.version.hip, "torch": torch.__version__,
            "source_sha256_16": source_hash(), "git_head": head}


def _entropy_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in ("paper_2608_15592_amd/csrc/entropy.hip", "paper_2608_15592_amd/csrc/estp_common.h"):
        h.update(open(os.path.join(ROOT, f), "rb").read())
    return h.hexdigest()[:16]


def _recorded_line(workload: str, fname: str, pattern: str):
    """Fields of the machine-readable line of a committed rocprofv3 summary, or None when the
    summary is for another workload or was taken on a different entropy-kernel source."""
    import re
    if workload != "llama":
        return None
    try:
        txt = open(os.path.join(ROOT, "profiles", fname)).read()
    except OSError:
        return None
    m = re.search(pattern + r" source_sha256_16=([0-9a-f]+)", txt)
    if not m or m.group(m.lastindex) != _entropy_source_hash():
        return None
    return m.groups()[:-1]


def recorded_traffic(workload: str):
    """HBM bytes per launch of the entropy kernel (calibrated FETCH_SIZE + WRITE_SIZE)."""
    g = _recorded_line(workload, "llama_path_hbm_counters.md", r"entropy_gemm traffic_bytes=(\d+)")
    return float(g[0]) if g else None


def recorded_clock(workload: str):
    """(sustained core clock in GHz, matrix-pipe busy fraction) of the entropy kernel, from the
    GRBM_GUI_ACTIVE / SQ_VALU_MFMA_BUSY_CYCLES counter summary."""
    g = _recorded_line(workload, "entropy_gemm_llama_clock_mfma_busy.md",
                       r"entropy_gemm sustained_clock_mhz=([0-9.]+) mfma_busy=([0-9.]+)")
    return (float(g[0]) / 1000.0, float(g[1])) if g else None


class HipEvent:
    """A HIP event recorded on the launch stream for timing only: created with
    hipEventDisableSystemFence, so recording it does not write back and invalidate the
    caches (the default event's system-scope fence adds ~6 us of idle time around every
    call it brackets and cools the cache for the next kernel).  The HIP runtime is the one
    torch already loaded."""
    _hip = None
    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self):
        import ctypes
        if HipEvent._hip is None:
            hip = ctypes.CDLL("libamdhip64.so.7")
            hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
            hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
            HipEvent._hip = hip
        self._ev = ctypes.c_void_p()
        rc = HipEvent._hip.hipEventCreateWithFlags(ctypes.byref(self._ev), self.DISABLE_SYSTEM_FENCE)
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed: {rc}")

    def record(self, stream):
        rc = HipEvent._hip.hipEventRecord(self._ev, ctypes_stream(stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed: {rc}")

    def elapsed_time(self, other: "HipEvent") -> float:
        import ctypes
        ms = ctypes.c_float()
        rc = HipEvent._hip.hipEventElapsedTime(ctypes.byref(ms), self._ev, other._ev)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed: {rc}")
        return float(ms.value)

    def __del__(self):
        if HipEvent._hip is not None and self._ev:
            HipEvent._hip.hipEventDestroy(self._ev)


def ctypes_stream(stream):
    import ctypes
    return ctypes.c_void_p(stream.cuda_stream)


def row_lse_torch(Q, K, cu_seqlens, scale, torch, rows: int = 1024):
    """Row log-sum-exps [L, Hq, n_tok] of every causal attention row, plain fp32 torch on the
    device, ``rows`` query rows at a time (stands in for what a FlashAttention-style prefill
    returns)."""
    L, n, Hq, _ = Q.shape
    G = Hq // K.shape[2]
    out = torch.empty(L, Hq, n, dtype=torch.float32, device=Q.device)
    for b in range(len(cu_seqlens) - 1):
        lo, hi = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        j = torch.arange(hi - lo, device=Q.device)[None, :]
        for l in range(L):
            k = K[l, lo:hi].float().repeat_interleave(G, dim=1).permute(1, 2, 0).contiguous()  # [Hq, dh, N]
            for i0 in range(0, hi - lo, rows):
                i1 = min(hi - lo, i0 + rows)
                q = Q[l, lo + i0:lo + i1].float().transpose(0, 1).contiguous()              # [Hq, r, dh]
                i = torch.arange(i0, i1, device=Q.device)[:, None]
                s = (torch.bmm(q, k) * scale).masked_fill(j > i, float("-inf"))
                out[l, :, lo + i0:lo + i1] = torch.logsumexp(s, dim=2)
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama", help="synthetic workload preset (synth.workloads)")
    ap.add_argument("--seed", type=int, default=42)
    ap.add_argument("--lambda1", type=float, default=0.5)
    ap.add_argument("--lambda2", type=float, default=0.5)
    ap.add_argument("--alpha", type=float, default=1.0)
    ap.add_argument("--norm", default="none", choices=["none", "zscore", "minmax"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true", help="also time the step captured in a HIP graph")
    ap.add_argument("--cpu-sample-prompts", type=int, default=2)
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run 3 device-to-device copies of BYTES (calibrates HBM byte counters)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(json.dumps({"error": "the path runs on one GPU: it is measured on one MI355X and has no "
                                   "multi-GPU sharding; run with --gpus 1"}))
        return 2

    import torch

    import paper_2608_15592_amd as estp
    from paper_2608_15592_amd.path import alloc_buffers
    import synth
    from synth import inputs as I

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_probe:
        a = torch.ones(args.copy_probe // 4, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": args.copy_probe, "copies": 3}), flush=True)
        return 0
    w = synth.get_workload(args.workload)
    log(f"workload {w.name}: {w.description}")
    t0 = time.time()
    inp = I.make_inputs(w, args.seed)
    n_tok = int(inp["n_tok"])
    B = len(inp["lengths"])
    max_len = int(inp["lengths"].max())
    log(f"inputs drawn in {time.time() - t0:.1f} s: n_tok={n_tok}, B={B}, max_seqlen={max_len}")
    t0 = time.time()
    X, W, Q, K = (to_dev(inp[k], torch) for k in ("X", "W", "Q", "K"))
    cu = to_dev(inp["cu_seqlens"], torch)
    Hdn, n_bins = w.head
    head = tuple(to_dev(inp[k], torch) for k in ("W1", "b1", "W2", "b2")) + (
        to_dev(inp["centres"], torch) if n_bins > 1 else None,)
    torch.cuda.synchronize()
    log(f"uploaded in {time.time() - t0:.1f} s")
    bufs = alloc_buffers(n_tok, B, max_len, w.d, w.V, w.L, w.Hq, w.Hkv, w.dh, Hdn, n_bins, X.device)
    stream = torch.cuda.current_stream()

    def step(evs=None, s=stream):
        if evs:
            evs[0].record(s)
        H = estp.token_entropy(X, W, H=bufs["H"], workspace=bufs["ws_entropy"], stream=s)
        if evs:
            evs[1].record(s)
        S = estp.attn_importance(Q, K, cu, max_len, S=bufs["S"], workspace=bufs["ws_importance"], stream=s)
        if evs:
            evs[2].record(s)
        pooled, _, _ = estp.combine_pool(X, S, H, cu, max_len, args.lambda1, args.lambda2, args.alpha, args.norm,
                                         pooled=bufs["pooled"], e=bufs["e"], top=bufs["top"],
                                         workspace=bufs["ws_pool"], stream=s)
        if evs:
            evs[3].record(s)
        estp.predict(pooled, *head, workspace=bufs["ws_predict"], stream=s)
        if evs:
            evs[4].record(s)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log(f"warmup step {i + 1}/{args.warmup} done")

    evs = [[HipEvent() for _ in range(5)] for _ in range(args.steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(args.steps):
        step(evs[i])
    stop.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    ms_per_step = total_ms / args.steps
    per_call = np.array([[e[k].elapsed_time(e[k + 1]) for k in range(4)] for e in evs])
    ent_ms, imp_ms, pool_ms, pred_ms = per_call.mean(axis=0)
    med_ms = np.median(per_call, axis=0)
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step "
        f"(entropy {ent_ms:.3f}, importance {imp_ms:.3f}, combine+pool {pool_ms:.3f}, head {pred_ms:.3f} ms)")

    # Side measurement: the same step captured once in a HIP graph and replayed (no launch gaps).
    graph_info = None
    if args.graph:
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):  # warm-up off the default stream before capture
            step(s=side)
        stream.wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step(s=torch.cuda.current_stream())
        torch.cuda.synchronize()
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        g0, g1 = HipEvent(), HipEvent()
        g0.record(stream)
        for _ in range(args.steps):
            g.replay()
        g1.record(stream)
        torch.cuda.synchronize()
        gms = g0.elapsed_time(g1) / args.steps
        graph_info = {"ms_per_step": gms, "tokens_per_s": n_tok / (gms * 1e-3), "eager_over_graph": ms_per_step / gms,
                      "note": "the timed step captured once in a HIP graph and replayed; not part of value"}
        del g
        log(f"graph replay: {gms:.3f} ms/step (eager {ms_per_step:.3f})")

    # The entropy call that also returns each token's most probable next token, timed on its own
    # against the plain call, interleaved (median of 3 each); its output goes to buffers of its own.
    am = torch.empty(n_tok, dtype=torch.int32, device=X.device)
    H_am = torch.empty(n_tok, dtype=torch.float32, device=X.device)
    estp.token_entropy(X, W, H=H_am, vocab_argmax=am, workspace=bufs["ws_entropy"], stream=stream)
    am_evs = [HipEvent() for _ in range(12)]
    for k in range(3):
        am_evs[4 * k].record(stream)
        estp.token_entropy(X, W, H=H_am, workspace=bufs["ws_entropy"], stream=stream)
        am_evs[4 * k + 1].record(stream)
        am_evs[4 * k + 2].record(stream)
        estp.token_entropy(X, W, H=H_am, vocab_argmax=am, workspace=bufs["ws_entropy"], stream=stream)
        am_evs[4 * k + 3].record(stream)
    torch.cuda.synchronize()
    plain_ms = float(np.median([am_evs[4 * k].elapsed_time(am_evs[4 * k + 1]) for k in range(3)]))
    am_ms = float(np.median([am_evs[4 * k + 2].elapsed_time(am_evs[4 * k + 3]) for k in range(3)]))
    del am, H_am
    log(f"entropy with next-token mode: {am_ms:.3f} ms (plain {plain_ms:.3f} ms)")

    # The one-pass importance call fed with a prefill's row log-sum-exps (here formed with plain
    # fp32 torch, untimed); timed on its own, outside the step.
    lse = row_lse_torch(Q, K, inp["cu_seqlens"], w.dh ** -0.5, torch)
    ws_lse = torch.empty(estp.load().estp_attn_importance_from_lse_workspace_size(n_tok, B, max_len, w.L, w.Hq, w.Hkv,
                                                                                 w.dh, 0),
                         dtype=torch.uint8, device=X.device)
    S_lse = torch.empty(n_tok, dtype=torch.float32, device=X.device)
    estp.attn_importance_from_lse(Q, K, lse, cu, max_len, S=S_lse, workspace=ws_lse, stream=stream)
    lse_evs = [HipEvent() for _ in range(6)]
    for k in range(5):
        lse_evs[k].record(stream)
        estp.attn_importance_from_lse(Q, K, lse, cu, max_len, S=S_lse, workspace=ws_lse, stream=stream)
    lse_evs[5].record(stream)
    torch.cuda.synchronize()
    lse_ms = float(np.mean([lse_evs[k].elapsed_time(lse_evs[k + 1]) for k in range(5)]))
    del lse, ws_lse, S_lse
    log(f"importance from prefill LSE: {lse_ms:.3f} ms (two-pass call {imp_ms:.3f} ms)")

    # One training step of a 16-bin head on the step's pooled vectors (Eq. 6-8, AdamW), timed on
    # its own: W1 [1024, d] dominates, read and written with its two moments.
    K_tr, Hd_tr = 16, 1024
    g_tr = torch.Generator(device="cpu").manual_seed(args.seed)
    n_par = Hd_tr * w.d + Hd_tr + K_tr * Hd_tr + K_tr
    theta = (torch.randn(n_par, generator=g_tr) * 0.02).to(X.device)
    m_tr, v_tr = torch.zeros_like(theta), torch.zeros_like(theta)
    edges = torch.cat([torch.zeros(1), torch.logspace(6, 14, K_tr, base=2.0)]).to(X.device)
    centres = 0.5 * (edges[1:] + edges[:-1])
    y_tr = torch.exp(torch.empty(B).uniform_(math.log(16.0), math.log(16384.0), generator=g_tr)).to(X.device)
    pooled_tr = bufs["pooled"]
    estp.head_train_step(pooled_tr, y_tr, edges, centres, theta, m_tr, v_tr, Hd_tr, 1, 0.5, 1e-4, stream=stream)
    tr_evs = [HipEvent() for _ in range(11)]
    for k in range(10):
        tr_evs[k].record(stream)
        estp.head_train_step(pooled_tr, y_tr, edges, centres, theta, m_tr, v_tr, Hd_tr, k + 2, 0.5, 1e-4,
                             stream=stream)
    tr_evs[10].record(stream)
    torch.cuda.synchronize()
    tr_ms = float(np.mean([tr_evs[k].elapsed_time(tr_evs[k + 1]) for k in range(10)]))
    tr_bytes = 6 * 4 * n_par + 4 * B * w.d
    del theta, m_tr, v_tr
    log(f"head training step (B={B}, {w.d}->{Hd_tr}->{K_tr}): {tr_ms:.3f} ms")

    # The Fig. 1b split on this step's H and S, and the padding of SJF batches of 16 built from
    # the step's predicted lengths against synthetic true lengths; timed on their own.
    H_s, S_s = bufs["H"], bufs["S"]
    yhat_s = estp.predict(bufs["pooled"], *head, workspace=bufs["ws_predict"], stream=stream)
    y_true = torch.exp(torch.empty(B).uniform_(math.log(16.0), math.log(16384.0), generator=g_tr)).to(
        torch.int32).to(X.device)
    an_evs = [HipEvent() for _ in range(3)]
    an_evs[0].record(stream)
    counts = estp.misalignment(H_s, S_s, cu, stream=stream)
    an_evs[1].record(stream)
    pad = estp.sjf_padding(y_true, yhat_s[2], 16, stream=stream)
    an_evs[2].record(stream)
    torch.cuda.synchronize()
    c = counts.sum(dim=0).tolist()
    pad = pad.tolist()
    analyses = {"misalignment_ms": an_evs[0].elapsed_time(an_evs[1]),
                "high_H_low_S_ratio": c[1] / max(1, c[0]), "low_H_high_S_ratio": c[3] / max(1, c[2]),
                "sjf_padding_ms": an_evs[1].elapsed_time(an_evs[2]), "sjf_padding_ratio": pad[0] / max(1, pad[1]),
                "note": "40% rank split per prompt on this step's H and S (synthetic inputs); SJF batches of 16 "
                        "ordered by the predicted lengths, synthetic true lengths"}
    log(f"analyses: misalignment {analyses['misalignment_ms']:.3f} ms, sjf padding {analyses['sjf_padding_ms']:.3f} ms")

    # A plain device-to-device copy of X, the bandwidth the pooling call is set against.
    Xc = torch.empty_like(X)
    Xc.copy_(X)
    cp_evs = [HipEvent() for _ in range(6)]
    for k in range(5):
        cp_evs[k].record(stream)
        Xc.copy_(X)
    cp_evs[5].record(stream)
    torch.cuda.synchronize()
    copy_ms = float(np.median([cp_evs[k].elapsed_time(cp_evs[k + 1]) for k in range(5)]))
    copy_gbps = 2 * X.numel() * X.element_size() / (copy_ms * 1e-3) / 1e9
    del Xc

    # The pooling call with cold caches: 1 GiB streamed through the caches before every
    # repetition, each call bracketed on its own (median of 5).  Read-flushed: a reduction over
    # the buffer leaves only clean lines, so the 256 MB MALL and the L2s hold none of X, H, S
    # and nothing is waiting to be written back.  Write-flushed: a fill of the buffer instead,
    # whose dirty lines (up to the MALL's 256 MB) are written back while the call reads X.
    flush = torch.zeros(1 << 28, dtype=torch.float32, device=X.device)
    torch.cuda.synchronize()

    def cold_pool(refill):
        times = []
        for k in range(6):
            if refill:
                flush.fill_(float(k))
            else:
                flush.sum()
            c0, c1 = HipEvent(), HipEvent()
            c0.record(stream)
            estp.combine_pool(X, bufs["S"], bufs["H"], cu, max_len, args.lambda1, args.lambda2, args.alpha,
                              args.norm, pooled=bufs["pooled"], e=bufs["e"], top=bufs["top"],
                              workspace=bufs["ws_pool"], stream=stream)
            c1.record(stream)
            torch.cuda.synchronize()
            if k:
                times.append(c0.elapsed_time(c1))
        return float(np.median(times))

    cold_ms = cold_pool(refill=False)
    cold_w_ms = cold_pool(refill=True)
    del flush

    ent_flop = 2.0 * n_tok * w.V * w.d
    imp_flop_alg = float(sum(int(T) * int(T) for T in inp["lengths"])) * w.dh * w.Hq * w.L  # one causal QK^T
    imp_exps = 2.0 * float(sum(int(T) * (int(T) + 1) // 2 for T in inp["lengths"])) * w.Hq * w.L  # two passes
    pool_bytes = n_tok * w.d * 2 + n_tok * 4 + B * w.d * 4
    ent_tflops = ent_flop / (ent_ms * 1e-3) / 1e12
    pool_gbps = pool_bytes / (pool_ms * 1e-3) / 1e9
    clock = recorded_clock(args.workload)
    f32 = w.dtype == "f32"  # fp32 inputs run the fp32 (VALU) kernels
    peak = PEAK_F32_TFLOPS if f32 else PEAK_BF16_TFLOPS
    result = {
        "metric": METRIC,
        "value": n_tok / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if f32 else "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.description,
            "n_tok": n_tok, "prompts": B, "d": w.d, "V": w.V, "Hq": w.Hq, "Hkv": w.Hkv, "dh": w.dh, "layers": w.L,
            "lambda1": args.lambda1, "lambda2": args.lambda2, "alpha": args.alpha, "norm": args.norm,
            "head": f"{w.d}->{Hdn}->{n_bins}",
        },
        "roofline": {
            "kernel": ("entropy_f32_kernel" if f32 else "entropy_gemm_kernel")
                      + " (+ entropy_merge_kernel inside the timed call)",
            "bound": "alu" if f32 else "mfma",
            "achieved": ent_tflops,
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": ent_tflops / peak,
            "traffic": recorded_traffic(args.workload),
            "work_per_launch": f"2*n_tok*V*d = {ent_flop:.4g} FLOP",
            # from the committed GRBM_GUI_ACTIVE / SQ_VALU_MFMA_BUSY_CYCLES summary of this kernel source
            "counter_run_clock_GHz": clock[0] if clock else None,
            "counter_run_mfma_busy": clock[1] if clock else None,
            "clock_note": "core clock and matrix-pipe busy of this kernel from GRBM_GUI_ACTIVE and "
                          "SQ_VALU_MFMA_BUSY_CYCLES in a separate counter run (profiles/), possibly on another box: "
                          "boxes differ by up to ~6% in the clock they sustain. The chip is power-limited under this "
                          "load, and the nominal peak assumes 2.4 GHz",
        },
        "kernels_ms": {"token_entropy": ent_ms, "attn_importance": imp_ms, "combine_pool": pool_ms,
                       "predict": pred_ms},
        "kernels_ms_median": dict(zip(("token_entropy", "attn_importance", "combine_pool", "predict"),
                                      (float(v) for v in med_ms))),
        "importance": {"alg_flop": imp_flop_alg, "alg_tflops": imp_flop_alg / (imp_ms * 1e-3) / 1e12,
                       "executed_tflops": 2 * imp_flop_alg / (imp_ms * 1e-3) / 1e12,
                       # each causal score is exponentiated once per pass; v_exp_f32 issues at a quarter of
                       # the FMA rate: 256 CUs x 4 SIMDs x 16 lanes / 4 x 2.4 GHz
                       "exp_roofline": {"bound": "alu", "exps": imp_exps, "achieved": imp_exps / (imp_ms * 1e-3),
                                        "peak": PEAK_EXP_PER_S, "unit": "exp/s",
                                        "frac": imp_exps / (imp_ms * 1e-3) / PEAK_EXP_PER_S}},
        "entropy_with_vocab_argmax": {"ms": am_ms, "plain_ms": plain_ms, "overhead": am_ms / plain_ms - 1.0,
                                      "note": "estp_token_entropy with the vocab_argmax output against the plain "
                                              "call, interleaved, median of 3 each; not part of the timed step"},
        "importance_from_prefill_lse": {"ms": lse_ms, "vs_two_pass": lse_ms / imp_ms,
                                        "note": "estp_attn_importance_from_lse with given row LSEs; not part of "
                                                "the timed step"},
        "head_train_step": {"ms": tr_ms, "head": f"{w.d}->{Hd_tr}->{K_tr}", "batch": B, "param_bytes_rw": tr_bytes,
                            "achieved_GBps": tr_bytes / (tr_ms * 1e-3) / 1e9,
                            "note": "estp_head_train_step (Eq. 8 loss, backward, AdamW); not part of the timed step"},
        "analyses": analyses,
        "pooling": {"bound": "hbm", "alg_bytes": pool_bytes, "achieved": pool_gbps, "peak": PEAK_HBM_GBPS,
                    "unit": "GB/s", "frac": pool_gbps / PEAK_HBM_GBPS,
                    "device_copy_GBps": copy_gbps, "frac_of_device_copy": pool_gbps / copy_gbps,
                    "cold_mall_ms": cold_ms, "cold_mall_GBps": pool_bytes / (cold_ms * 1e-3) / 1e9,
                    "cold_mall_frac": pool_bytes / (cold_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS,
                    "after_write_flush_ms": cold_w_ms,
                    "after_write_flush_GBps": pool_bytes / (cold_w_ms * 1e-3) / 1e9,
                    "note": "whole combine_pool call (weights + pooling); in the step, X is not cache resident "
                            "(importance streams Q and K just before); cold_mall_*: median of 5 calls, each after "
                            "a 1 GiB read that evicts everything with clean lines; after_write_flush_*: each after a "
                            "1 GiB write, whose dirty lines are written back during the call; device copy counts "
                            "read + write bytes"},
        "device": build_info(torch),
        **({"graph": graph_info} if graph_info else {}),
    }
    if not args.no_cpu_baseline:
        log("timing the fp64 oracle on the host sample ...")
        result["cpu_baseline"], ref, n_ref = cpu_baseline(inp, args.lambda1, args.lambda2, args.alpha, args.norm,
                                                          args.cpu_sample_prompts)
        log(f"oracle: {result['cpu_baseline']['value']:.1f} tokens/s")
        got = {k: bufs[k].cpu().numpy() for k in ("H", "S", "pooled", "top")}
        got["yhat"] = yhat_s[0].cpu().numpy()
        result["parity"] = parity_of_run(ref, n_ref, got)
        log(f"parity of this run on the oracle sample: {result['parity']}")
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
