"""HiLS attention benchmark on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-decode] [--no-train] [--no-cpu]

A step is one pass of the operator over one batch of synthetic input.  The
headline workload is 32K-token causal prefill in bf16 (B=1, Hq=32, Hkv=8,
d=128, chunk 64, top-16, window 512): every row of the path runs -- landmark
scoring, group max, top-K selection, local-window attention, per-chunk
attention and the fusion epilogue.  ``value`` is prefill tokens/s with all
inputs resident in HBM.  Decode (32 x 131K-token caches) and fwd+bwd at
4 x 16K are reported beside it in ``extra``.

Timing uses HIP events on the stream the library launches on: every step is
bracketed by two events and the reported step time is the median over the
timed steps (the mean is given beside it); the library's optional per-kernel
timing mode brackets every kernel launch in a second pass over the same
number of steps.  The roofline object describes the dominant kernel (largest
total time): its average launch duration against the method's work in that
kernel -- FLOPs of the selected pairs and the causal band only, bytes of the
method's inputs read once and outputs written once -- under whichever bound
is tighter (bf16 MFMA for the prefill kernels).  Bytes the design adds (the
chunk pass's per-slot records) are not method bytes: they appear in the
rocprofv3 traffic and its ratio to the method bytes.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
METRIC = "HiLS attn tokens/s + decode HBM GB/s & prefill MFMA util vs MI355X peak"
# The paper's own efficiency figures (Sec. 7.1, Fig. 5): end-to-end latencies of a
# 345M-parameter model (16 layers, 16 query / 2 KV heads, d = 64; S = 64, K = 32,
# W = 512) served by SGLang with Triton kernels on one NVIDIA H800, bf16, batch 1.
# Context only: whole-model latencies on other hardware, not operator figures.
PAPER_CONTEXT = {"hardware": "1x NVIDIA H800", "model": "345M, 16 layers, 16/2 heads, d 64",
                 "prefill_512k_latency_s": {"hils": 5.0, "full_attention": 67.0},
                 "decode_512k_ms_per_token": {"hils": 5.5, "full_attention": 85.9},
                 "crossover_context_tokens": 16384,
                 "source": "Sec. 7.1 and Fig. 5 (end-to-end, SGLang + Triton)"}


def n_candidates(i, S, W):
    return np.maximum(0, (i - W + 1) // S)


def prefill_work(B, Hq, Hkv, N, d, S, K, W):
    """Algorithmic work of a causal prefill (selected pairs and the window only)."""
    i = np.arange(N, dtype=np.int64)
    ncand = n_candidates(i, S, W)
    nloc = i - ncand * S + 1
    nsel = np.minimum(K, ncand)
    attn_flops = B * Hq * 4 * d * float((nloc + S * nsel).sum())   # QK^T and PV, 2 flops per MAC
    score_flops = B * Hq * 2 * d * float(ncand.sum())                # landmark dot products
    return attn_flops, score_flops


def prefill_kernel_model(B, Hq, Hkv, N, L, d, S, K, W, elem=2):
    """Per-kernel method FLOPs and method bytes of one bf16 prefill launch (the
    design's own intermediates -- per-slot records, the inverse index -- are not
    counted; they show in the measured traffic).

    k_pf_score : landmark scores over C_i, 2d per (head, candidate); reads q and
                 the landmarks once, writes idx (the fused scorer).
    k_pf_sigma : the same scores and their group max, the split scorer's first
                 pass (the group-score array it writes is the design's).
    k_pf_select: the top-K of every row from the group scores: no method FLOPs;
                 writes idx.
    k_pf_chunks: per selected (row, head, chunk) QK^T + PV over S keys (4dS) and
                 the surrogate score (2d); reads q and the K/V once.
    k_pf_local : window QK^T + PV, 4d per (row, head, window key), and the fusion;
                 reads q and K/V once, writes out and lse.
    design_bytes: the records k_pf_chunks writes and k_pf_local reads back (the bf16
                 chunk output and the fp32 score per (row, head, slot)).
    """
    i = np.arange(N, dtype=np.int64)
    ncand = n_candidates(i, S, W)
    nloc = i - ncand * S + 1
    nsel = float(np.minimum(K, ncand).sum())
    qbytes = B * Hq * N * d * elem
    kvbytes = 2 * B * Hkv * L * d * elem
    lmkbytes = B * Hq * (L // S) * d * elem
    idxbytes = B * Hkv * N * K * 4
    records = B * Hq * nsel * (d * elem + 4)
    return {
        "k_pf_score": {"flop": B * Hq * 2 * d * float(ncand.sum()), "bytes": qbytes + lmkbytes + idxbytes},
        "k_pf_sigma": {"flop": B * Hq * 2 * d * float(ncand.sum()), "bytes": qbytes + lmkbytes,
                       "design_bytes": B * Hkv * 4 * float(ncand.sum())},
        "k_pf_select": {"flop": 0.0, "bytes": idxbytes, "design_bytes": B * Hkv * 4 * float(ncand.sum())},
        "k_pf_chunks": {"flop": B * Hq * (4 * d * S + 2 * d) * nsel, "bytes": qbytes + kvbytes,
                        "design_bytes": records},
        "k_pf_local": {"flop": B * Hq * 4 * d * float(nloc.sum()), "bytes": qbytes + kvbytes + qbytes + B * Hq * N * 4,
                       "design_bytes": records},
    }


def prefill_method_bytes(B, Hq, Hkv, N, L, d, S, K, elem=2):
    """Bytes the whole prefill must move at least: q, k, v, landmarks read once;
    out, lse, idx written once."""
    return (2 * B * Hq * N * d + 2 * B * Hkv * L * d + B * Hq * (L // S) * d) * elem + B * Hq * N * 4 + \
        B * Hkv * N * K * 4


def decode_bytes(B, Hq, Hkv, Hl, ctx, d, S, K, W, elem=2, N=1):
    """Algorithmic HBM bytes of one decode step of N new queries per sequence (the
    last at position ctx + N - 1): landmark scan over C_i (once), the K retrieved
    chunks' K/V of every query, the local window's K/V (once), q in, out + lse out."""
    i = ctx + N - 1
    ncand = int(n_candidates(np.array(i), S, W))
    nloc = i - ncand * S + 1
    lmk = B * Hl * ncand * d * elem
    kv = B * Hkv * (N * min(K, ncand) * S + nloc) * d * elem * 2
    qo = N * (B * Hq * d * elem * 2 + B * Hq * 4)
    return lmk + kv + qo, dict(landmarks=lmk, kv=kv, q_out=qo)


def source_sha(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def load_traffic(kernel_tag):
    """HBM traffic per launch from committed rocprofv3 --pmc counters, or None
    when no counters exist or the kernel source changed since they were taken."""
    p = os.path.join(ROOT, "profiles", f"{kernel_tag}_pmc.json")
    if not os.path.exists(p):
        return None
    rec = json.load(open(p))
    src = os.path.join(ROOT, rec["source"])
    if not os.path.exists(src) or source_sha(src) != rec["source_sha"]:
        return None
    return rec["bytes_per_dispatch"]


def measured_peaks(torch):
    """What this machine sustains with plain library kernels: a 1 GiB device copy
    (torch's copy kernel, bytes read + written) and an 8192^3 bf16 GEMM
    (hipBLASLt through torch.matmul).  Context for the published peaks."""
    x = torch.ones(2 ** 28, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    a = torch.randn(8192, 8192, dtype=torch.bfloat16, device="cuda")
    b = torch.randn(8192, 8192, dtype=torch.bfloat16, device="cuda")
    t = Timer(torch)
    copy_ms, _ = t.run(lambda: y.copy_(x), 20, 3)
    gemm_ms, _ = t.run(lambda: torch.matmul(a, b), 20, 3)
    out = {"copy_1gib_gbs": round(2 * x.numel() * 4 / (copy_ms * 1e-3) / 1e9, 1),
           "bf16_gemm_8192_tflops": round(2 * 8192 ** 3 / (gemm_ms * 1e-3) / 1e12, 1),
           "note": "torch copy kernel (read + write bytes) and hipBLASLt GEMM; published peaks: "
                   f"HBM {HBM_PEAK_GBS:.0f} GB/s, dense bf16 MFMA {BF16_MFMA_PEAK_TFLOPS:.0f} TFLOP/s"}
    del x, y, a, b
    torch.cuda.empty_cache()
    return out


class Timer:
    """HIP events on the current (library) stream around every step; returns the
    median and the mean step time in ms."""

    def __init__(self, torch):
        self.torch = torch

    def run(self, fn, steps, warmup, before=None):
        t = self.torch
        for _ in range(warmup):
            fn()
        t.cuda.synchronize()
        st = t.cuda.current_stream()
        ev = [(t.cuda.Event(enable_timing=True), t.cuda.Event(enable_timing=True)) for _ in range(steps)]
        for e0, e1 in ev:
            if before is not None:
                before()
            e0.record(st)
            fn()
            e1.record(st)
        t.cuda.synchronize()
        ms = sorted(e0.elapsed_time(e1) for e0, e1 in ev)
        return float(np.median(ms)), float(np.mean(ms))


def chunk_overlap(idx, M=16):
    """Normalised chunk overlap of blocks of M adjacent queries, (M K - |union|) / ((M - 1) K),
    over the blocks whose rows all hold K chunks (a statistic of the inputs)."""
    B, Hkv, N, K = idx.shape
    n0 = (N // M) * M
    blk = idx[:, :, :n0].reshape(B, Hkv, n0 // M, M * K)
    full = (blk >= 0).all(axis=-1)
    srt = np.sort(blk, axis=-1)
    uniq = 1 + (np.diff(srt, axis=-1) != 0).sum(axis=-1)
    vals = (M * K - uniq[full]) / ((M - 1) * K)
    return float(vals.mean()) if vals.size else float("nan")


def bench_prefill(torch, hils, synth, W_, steps, warmup, flags=0, rho=None):
    """Times `steps` prefill calls (HIP events on the library's stream, no
    per-kernel events), then a second pass with per-kernel timing for the
    breakdown; returns (params, host inputs, ms/step, kernels)."""
    p = hils.Params(B=W_.B, Hq=W_.Hq, Hkv=W_.Hkv, N=W_.N, L=W_.L, d=W_.d, chunk=W_.chunk, topk=W_.topk,
                    window=W_.window, dtype=W_.dtype, flags=flags)
    nc = p.L // p.chunk
    dt = p.torch_dtype
    host = {
        "q": synth.normal_host((p.B, p.Hq, p.N, p.d), synth.seed_for(W_.wid, "q"), p.dtype),
        "k": synth.normal_host((p.B, p.Hkv, p.L, p.d), synth.seed_for(W_.wid, "k"), p.dtype),
        "v": synth.normal_host((p.B, p.Hkv, p.L, p.d), synth.seed_for(W_.wid, "v"), p.dtype),
        "lmk": synth.normal_host((p.B, p.Hq, nc, p.d), synth.seed_for(W_.wid, "lmk"), p.dtype),
    }
    dev = {k: v.to("cuda", dt).contiguous() for k, v in host.items()}
    if rho is not None:  # queries correlated along the sequence (the locality inputs)
        dev["q"] = synth.ar1_host((p.B, p.Hq, p.N, p.d), synth.seed_for(W_.wid, "q"), p.dtype, rho=rho,
                                  device="cuda").to(dt).contiguous()
    out = torch.empty(p.B, p.Hq, p.N, p.d, dtype=dt, device="cuda")
    lse = torch.empty(p.B, p.Hq, p.N, dtype=torch.float32, device="cuda")
    idx = torch.empty(p.B, p.Hkv, p.N, p.topk, dtype=torch.int32, device="cuda")
    ws = torch.empty(max(1, hils.hils_workspace_size(p, hils.HILS_OP_PREFILL)), dtype=torch.uint8, device="cuda")

    def step():
        hils.hils_prefill_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"], out=out, lse=lse, idx=idx, workspace=ws)

    ms, ms_mean = Timer(torch).run(step, steps, warmup)
    hils.hils_timing_enable(True)
    Timer(torch).run(step, steps, 0)
    kernels = hils.hils_timing_read()
    hils.hils_timing_enable(False)
    for k in kernels.values():
        k["avg_ms"] = k["total_ms"] / max(1, k["launches"])
    p.overlap16 = chunk_overlap(idx.cpu().numpy(), 16) if p.topk <= 64 and p.dtype == "bf16" else float("nan")
    p.ms_mean = ms_mean
    del dev, ws
    torch.cuda.empty_cache()
    return p, host, ms, kernels


def bench_decode(torch, hils, synth, W_, steps, warmup, paged=False, N=1, flags=0, Hl=0):
    """One decode step of N new queries per sequence after W_.ctx cached tokens.
    paged: the caches are pools of one-chunk pages in a seeded random order (a
    random permutation as the page table).  Hl: landmark heads (0: Hq)."""
    p = hils.Params(B=W_.B, Hq=W_.Hq, Hkv=W_.Hkv, N=N, L=W_.L, d=W_.d, chunk=W_.chunk, topk=W_.topk,
                    window=W_.window, dtype=W_.dtype, flags=flags, Hl=Hl)
    Hl = Hl or p.Hq
    nc = p.L // p.chunk
    if paged:
        P = p.B * nc
        gen = torch.Generator(device="cpu")
        gen.manual_seed(synth.seed_for(W_.wid, "page_table"))
        table = torch.randperm(P, generator=gen).to(torch.int32).reshape(p.B, nc).cuda()
        kv_shape, lmk_shape = (P, p.Hkv, p.chunk, p.d), (P, Hl, p.d)
    else:
        kv_shape, lmk_shape = (p.B, p.Hkv, p.L, p.d), (p.B, Hl, nc, p.d)
    dev = {
        "q": synth.normal_device((p.B, p.Hq, N, p.d), synth.seed_for(W_.wid, "q"), p.dtype, "cuda"),
        "k": synth.normal_device(kv_shape, synth.seed_for(W_.wid, "k"), p.dtype, "cuda"),
        "v": synth.normal_device(kv_shape, synth.seed_for(W_.wid, "v"), p.dtype, "cuda"),
        "lmk": synth.normal_device(lmk_shape, synth.seed_for(W_.wid, "lmk"), p.dtype, "cuda"),
    }
    seqlens = torch.full((p.B,), W_.ctx + N, dtype=torch.int32, device="cuda")
    out = torch.empty(p.B, p.Hq, N, p.d, dtype=p.torch_dtype, device="cuda")
    lse = torch.empty(p.B, p.Hq, N, dtype=torch.float32, device="cuda")
    idx = torch.empty(p.B, p.Hkv, N, p.topk, dtype=torch.int32, device="cuda")
    ws = torch.empty(max(1, hils.hils_workspace_size(p, hils.HILS_OP_DECODE)), dtype=torch.uint8, device="cuda")
    # reading 1 GiB between steps evicts L2 and MALL with clean lines, so the
    # timed step streams from HBM without paying for dirty write-backs
    flush = torch.ones(2 ** 28, dtype=torch.float32, device="cuda")
    sink = torch.empty((), dtype=torch.float32, device="cuda")

    def step():
        if paged:
            hils.hils_decode_paged_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"], table, seqlens=seqlens, out=out,
                                       lse=lse, idx=idx, workspace=ws)
        else:
            hils.hils_decode_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"], seqlens=seqlens, out=out, lse=lse,
                                 idx=idx, workspace=ws)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()

    def timed(instrumented):
        hils.hils_timing_enable(instrumented)
        med, mean = Timer(torch).run(step, steps, 0, before=lambda: torch.sum(flush, dim=0, out=sink))
        kern = hils.hils_timing_read() if instrumented else None
        hils.hils_timing_enable(False)
        return med, mean, kern

    # the step time is taken without per-kernel events (they add a few us per
    # launch to a ~0.2 ms step); a second, instrumented pass gives the breakdown
    ms, ms_mean, _ = timed(False)
    _, _, kernels = timed(True)
    nbytes, parts = decode_bytes(p.B, p.Hq, p.Hkv, Hl, W_.ctx, p.d, p.chunk, p.topk, p.window, N=N)
    del dev, flush, sink
    torch.cuda.empty_cache()
    return {"workload": W_.name, "paged": paged, "new_tokens_per_seq": N, "landmark_heads": Hl,
            "ms_per_step": round(ms, 4), "ms_per_step_mean": round(ms_mean, 4), "steps": steps,
            "tokens_per_s": round(p.B * N / (ms * 1e-3), 1),
            "algorithmic_bytes": nbytes, "bytes_breakdown": parts,
            "hbm_gbs": round(nbytes / (ms * 1e-3) / 1e9, 1),
            "frac_hbm_peak": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "kernels_avg_ms": {k: round(v["total_ms"] / max(1, v["launches"]), 4) for k, v in kernels.items()}}


def bench_train(torch, hils, synth, W_, steps, warmup):
    p = hils.Params(B=W_.B, Hq=W_.Hq, Hkv=W_.Hkv, N=W_.N, L=W_.L, d=W_.d, chunk=W_.chunk, topk=W_.topk,
                    window=W_.window, dtype=W_.dtype)
    nc = p.L // p.chunk
    dev = {
        "q": synth.normal_device((p.B, p.Hq, p.N, p.d), synth.seed_for(W_.wid, "q"), p.dtype, "cuda"),
        "k": synth.normal_device((p.B, p.Hkv, p.L, p.d), synth.seed_for(W_.wid, "k"), p.dtype, "cuda"),
        "v": synth.normal_device((p.B, p.Hkv, p.L, p.d), synth.seed_for(W_.wid, "v"), p.dtype, "cuda"),
        "lmk": synth.normal_device((p.B, p.Hq, nc, p.d), synth.seed_for(W_.wid, "lmk"), p.dtype, "cuda"),
        "dout": synth.normal_device((p.B, p.Hq, p.N, p.d), synth.seed_for(W_.wid, "dout"), p.dtype, "cuda"),
    }
    ws = torch.empty(hils.hils_workspace_size(p, hils.HILS_OP_BWD), dtype=torch.uint8, device="cuda")

    def step():
        out, lse, idx = hils.hils_prefill_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"])
        hils.hils_bwd(p, dev["dout"], dev["q"], dev["k"], dev["v"], dev["lmk"], out, lse, idx, workspace=ws)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ms, ms_mean = Timer(torch).run(step, steps, 0)
    hils.hils_timing_enable(True)
    Timer(torch).run(step, steps, 0)
    kernels = hils.hils_timing_read()
    hils.hils_timing_enable(False)
    attn, score = prefill_work(p.B, p.Hq, p.Hkv, p.N, p.d, p.chunk, p.topk, p.window)
    fwd = attn + score
    bwd = 2.5 * attn + 2 * score  # dq, dk, dv recompute: 10d vs 4d per attended pair; score grads
    del dev
    torch.cuda.empty_cache()
    return {"workload": W_.name, "ms_per_step": round(ms, 3), "ms_per_step_mean": round(ms_mean, 3), "steps": steps,
            "tokens_per_s": round(p.B * p.N / (ms * 1e-3), 1),
            "algorithmic_tflop": round((fwd + bwd) / 1e12, 3),
            "mfma_frac_useful": round((fwd + bwd) / (ms * 1e-3) / 1e12 / BF16_MFMA_PEAK_TFLOPS, 5),
            "kernels_avg_ms": {k: round(v["total_ms"] / max(1, v["launches"]), 3) for k, v in kernels.items()}}


def bench_landmark(torch, hils, synth, W_, steps, warmup):
    """Landmark compression (Prop. 3.1) forward and backward on the workload's
    K, one landmark per (query head, chunk).  Algorithmic bytes: the forward
    reads K and q' and writes k' and b'; the backward reads K, q', dk' and db'
    and writes dq' and dK."""
    p = hils.Params(B=W_.B, Hq=W_.Hq, Hkv=W_.Hkv, N=1, L=W_.L, d=W_.d, chunk=W_.chunk, topk=1, window=1,
                    dtype=W_.dtype)
    nc, Hl, e = p.L // p.chunk, p.Hq, 2 if p.dtype == "bf16" else 4
    lq = synth.normal_device((p.B, Hl, nc, p.d), synth.seed_for(W_.wid, "lmk"), p.dtype, "cuda")
    k = synth.normal_device((p.B, p.Hkv, p.L, p.d), synth.seed_for(W_.wid, "k"), p.dtype, "cuda")
    dl = synth.normal_device((p.B, Hl, nc, p.d), synth.seed_for(W_.wid, "dout"), p.dtype, "cuda")
    db = synth.normal_device((p.B, Hl, nc), synth.seed_for(W_.wid, "bias"), "f32", "cuda")
    lmk, bias = hils.hils_landmark_fwd(p, lq, k)
    dlq, dk = hils.hils_landmark_bwd(p, lq, k, dl, db)
    kb, lb, bb = p.B * p.Hkv * p.L * p.d * e, p.B * Hl * nc * p.d * e, p.B * Hl * nc * 4
    out = {"workload": W_.name, "landmark_heads": Hl}
    for name, fn, nbytes in (("fwd", lambda: hils.hils_landmark_fwd(p, lq, k, lmk, bias), kb + 2 * lb + bb),
                             ("bwd", lambda: hils.hils_landmark_bwd(p, lq, k, dl, db, dlq, dk), 2 * kb + 3 * lb + bb)):
        ms, _ = Timer(torch).run(fn, steps, warmup)
        out[name] = {"ms": round(ms, 4), "bytes": nbytes, "gbs": round(nbytes / (ms * 1e-3) / 1e9, 1),
                     "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    del lq, k, dl, db, lmk, bias, dlq, dk
    torch.cuda.empty_cache()
    return out


def cpu_baseline(W_, host, target_s=20.0):
    """The oracle (plain fp32 build, as it stands) on a bounded sample of query
    rows of the same workload, on all host cores; scaled to tokens/s."""
    import oracle

    threads = len(os.sched_getaffinity(0))
    os.environ.setdefault("OMP_NUM_THREADS", str(threads))
    threads = int(os.environ["OMP_NUM_THREADS"])
    s = oracle.Shape(B=W_.B, Hq=W_.Hq, Hkv=W_.Hkv, Hl=W_.Hq, N=W_.N, L=W_.L, d=W_.d, chunk=W_.chunk,
                     topk=W_.topk, window=W_.window, scale=float(np.float32(W_.scale)))
    arrs = {k: host[k].numpy() for k in ("q", "k", "v", "lmk")}
    nrows = 64
    while True:
        rows = np.stack([np.zeros(nrows, np.int64), np.linspace(0, W_.N - 1, nrows).astype(np.int64)], 1)
        t0 = time.perf_counter()
        oracle.fwd(s, arrs["q"], arrs["k"], arrs["v"], arrs["lmk"], rows=rows, prec="f32")
        dt = time.perf_counter() - t0
        if dt * threads >= target_s or nrows >= W_.N:
            break
        nrows = min(W_.N, int(nrows * max(2.0, min(16.0, target_s / max(dt * threads, 1e-3)))))
    model = "unknown CPU"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": round(nrows / dt, 2), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{nrows} query rows evenly spaced over the {W_.N}-token sequence (all {W_.Hq} heads), "
                      f"fp32 oracle, {dt:.2f} s wall on {threads} threads of a {model}"}


def run_part(part, torch, hils, synth, WORKLOADS, args):
    """One part of the bench on its own (each of its workloads as in the full run)."""
    Wp, Wd = WORKLOADS["prefill_32k_bf16"], WORKLOADS["decode_131k_bf16_b32"]
    out = {"part": part}
    if part == "prefill":
        _, _, ms, kt = bench_prefill(torch, hils, synth, Wp, args.steps, args.warmup)
        out[Wp.name] = {"ms_per_step": round(ms, 4), "kernels_avg_ms": {k: round(v["avg_ms"], 4) for k, v in kt.items()}}
    elif part == "decode":
        out["decode"] = bench_decode(torch, hils, synth, Wd, args.steps, args.warmup)
        out["decode_1m"] = bench_decode(torch, hils, synth, WORKLOADS["decode_1m_bf16_b4"], args.steps, args.warmup)
        out["decode_paged"] = bench_decode(torch, hils, synth, Wd, args.steps, args.warmup, paged=True)
        out["decode_4_new_tokens"] = bench_decode(torch, hils, synth, Wd, args.steps, args.warmup, N=4)
        out["decode_Hl_eq_Hkv"] = bench_decode(torch, hils, synth, Wd, args.steps, args.warmup, Hl=Wd.Hkv)
        out["decode_head_norm"] = bench_decode(torch, hils, synth, Wd, args.steps, args.warmup,
                                               flags=hils.HILS_FLAG_HEAD_NORM_SELECT)
    elif part == "train":
        out["train"] = bench_train(torch, hils, synth, WORKLOADS["train_16k_bf16_b4"], args.steps, args.warmup)
    elif part == "landmark":
        out["landmark"] = bench_landmark(torch, hils, synth, Wp, args.steps, args.warmup)
    elif part == "variants":
        U = hils.HILS_FLAG_UNION_PACKING
        for name, W_, fl, rho in (("prefill_head_norm", Wp, hils.HILS_FLAG_HEAD_NORM_SELECT, None),
                                  ("prefill_mha_G1", Wp.with_(Hkv=Wp.Hq), 0, None),
                                  ("prefill_union_packing", Wp, U, None),
                                  ("prefill_locality_chunk_major", Wp, 0, 0.97),
                                  ("prefill_locality_union_packing", Wp, U, 0.97)):
            pv, _, msv, kv = bench_prefill(torch, hils, synth, W_, args.steps, args.warmup, flags=fl, rho=rho)
            out[name] = {"ms_per_step": round(msv, 4), "chunk_overlap_16": round(pv.overlap16, 4),
                         "kernels_avg_ms": {k: round(v["avg_ms"], 4) for k, v in kv.items()}}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-train", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-landmark", action="store_true")
    ap.add_argument("--no-variants", action="store_true")
    ap.add_argument("--part", default="all", choices=["all", "prefill", "decode", "train", "landmark", "variants"],
                    help="run one part only and print its JSON (for per-workload profiles); the contract "
                         "line is printed by the default, all")
    ap.add_argument("--copy-probe", action="store_true",
                    help="first copy 1 GiB device-to-device (a plain copy kernel of known size, used to "
                         "calibrate rocprofv3 FETCH_SIZE/WRITE_SIZE)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU only (the operator has no multi-GPU path); "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2607_02980_amd import hils, synth
    from paper_2607_02980_amd.configs import WORKLOADS

    torch.cuda.set_device(0)
    if args.copy_probe:
        x = torch.ones(2 ** 28, dtype=torch.float32, device="cuda")
        y = x.clone()
        torch.cuda.synchronize()
        del x, y
    Wp = WORKLOADS["prefill_32k_bf16"]
    if args.part != "all":
        print(json.dumps(run_part(args.part, torch, hils, synth, WORKLOADS, args)), flush=True)
        return
    p, host, ms, kernels = bench_prefill(torch, hils, synth, Wp, args.steps, args.warmup)
    model = prefill_kernel_model(p.B, p.Hq, p.Hkv, p.N, p.L, p.d, p.chunk, p.topk, p.window)
    table = {}
    for name, k in kernels.items():
        row = {"avg_ms": round(k["avg_ms"], 4), "launches": k["launches"]}
        if name in model:
            t = k["avg_ms"] * 1e-3
            f, b = model[name]["flop"], model[name]["bytes"]
            row.update({"method_flop": f, "method_bytes": b, "tflops": round(f / t / 1e12, 2),
                        "mfma_frac": round(f / t / 1e12 / BF16_MFMA_PEAK_TFLOPS, 4),
                        "method_gbs": round(b / t / 1e9, 1), "hbm_frac_method": round(b / t / 1e9 / HBM_PEAK_GBS, 4),
                        "bound": "mfma" if f / (BF16_MFMA_PEAK_TFLOPS * 1e12) >= b / (HBM_PEAK_GBS * 1e9) else "hbm"})
            if "design_bytes" in model[name]:
                row["design_bytes"] = model[name]["design_bytes"]
            tr = load_traffic(f"{name}_{Wp.name}")
            if tr is not None:
                row.update({"traffic": tr, "traffic_gbs": round(tr / t / 1e9, 1),
                            "traffic_over_method_bytes": round(tr / b, 2)})
        table[name] = row
    dom = max((n for n in table if n in model), key=lambda n: kernels[n]["total_ms"])
    d = table[dom]
    if d["bound"] == "mfma":
        achieved, peak, unit = d["tflops"], BF16_MFMA_PEAK_TFLOPS, "TFLOP/s"
    else:
        achieved, peak, unit = d["method_gbs"], HBM_PEAK_GBS, "GB/s"
    attn_flops, score_flops = prefill_work(p.B, p.Hq, p.Hkv, p.N, p.d, p.chunk, p.topk, p.window)
    traffic = load_traffic(f"{dom}_{Wp.name}")
    mbytes = prefill_method_bytes(p.B, p.Hq, p.Hkv, p.N, p.L, p.d, p.chunk, p.topk)
    res = {
        "metric": METRIC, "value": round(p.B * p.N / (ms * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": Wp.name, "B": p.B, "Hq": p.Hq, "Hkv": p.Hkv, "d": p.d, "seq_len": p.N,
                   "chunk": p.chunk, "topk": p.topk, "window": p.window, "landmark_heads": p.Hq},
        "roofline": {"bound": d["bound"], "kernel": dom, "achieved": achieved, "peak": peak, "unit": unit,
                     "frac": round(achieved / peak, 5), "traffic": traffic,
                     "traffic_over_method_bytes": round(traffic / d["method_bytes"], 2) if traffic else None,
                     "per_launch": {"method_flop": d["method_flop"], "method_bytes": d["method_bytes"],
                                    "design_bytes": d.get("design_bytes")},
                     "hbm_on_method_bytes": {"gbs": d["method_gbs"], "frac": d["hbm_frac_method"]},
                     "kernel_avg_ms": d["avg_ms"]},
        "extra": {"ms_per_step_mean": round(p.ms_mean, 4),
                  "prefill_kernels": table,
                  "prefill_useful_mfma_frac": round((attn_flops + score_flops) / (ms * 1e-3) / 1e12
                                                    / BF16_MFMA_PEAK_TFLOPS, 5),
                  "prefill_method_bytes": mbytes,
                  "prefill_hbm_frac_on_method_bytes": round(mbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 5),
                  "paper_context": PAPER_CONTEXT},
    }
    del p
    torch.cuda.empty_cache()
    if not args.no_decode:
        Wd = WORKLOADS["decode_131k_bf16_b32"]
        res["extra"]["decode"] = bench_decode(torch, hils, synth, Wd, args.steps, args.warmup)
        res["extra"]["decode_1m"] = bench_decode(torch, hils, synth, WORKLOADS["decode_1m_bf16_b4"], args.steps, args.warmup)
        res["extra"]["decode_paged"] = bench_decode(torch, hils, synth, Wd, args.steps, args.warmup, paged=True)
        res["extra"]["decode_4_new_tokens"] = bench_decode(torch, hils, synth, Wd, args.steps, args.warmup, N=4)
        res["extra"]["decode_Hl_eq_Hkv"] = bench_decode(torch, hils, synth, WORKLOADS["decode_131k_bf16_b32"],
                                                        args.steps, args.warmup, Hl=WORKLOADS["decode_131k_bf16_b32"].Hkv)
    if not args.no_train:
        res["extra"]["train"] = bench_train(torch, hils, synth, WORKLOADS["train_16k_bf16_b4"], args.steps, args.warmup)
    # the tiny fp32 workload (2K tokens, 4/1 heads, d 64, top-4): latency of one prefill
    Wt = WORKLOADS["prefill_2k_f32_tiny"]
    pt, _, mst, kt = bench_prefill(torch, hils, synth, Wt, args.steps, args.warmup)
    res["extra"]["prefill_2k_f32_tiny"] = {"ms_per_step": round(mst, 4), "ms_per_step_mean": round(pt.ms_mean, 4),
                                           "tokens_per_s": round(pt.B * pt.N / (mst * 1e-3), 1),
                                           "kernels_avg_ms": {k: round(v["avg_ms"], 4) for k, v in kt.items()}}
    res["extra"]["measured_peaks"] = measured_peaks(torch)
    if not args.no_landmark:
        res["extra"]["landmark"] = bench_landmark(torch, hils, synth, Wp, args.steps, args.warmup)
    if not args.no_variants:
        # selection variants: per-head normalised ranking, and one query head per KV head (MHA)
        U = hils.HILS_FLAG_UNION_PACKING
        for name, W_, fl, rho in (("prefill_head_norm", Wp, hils.HILS_FLAG_HEAD_NORM_SELECT, None),
                                  ("prefill_mha_G1", Wp.with_(Hkv=Wp.Hq), 0, None),
                                  ("prefill_union_packing", Wp, U, None),
                                  ("prefill_locality_chunk_major", Wp, 0, 0.97),
                                  ("prefill_locality_union_packing", Wp, U, 0.97)):
            pv, _, msv, kv = bench_prefill(torch, hils, synth, W_, args.steps, args.warmup, flags=fl, rho=rho)
            res["extra"][name] = {"ms_per_step": round(msv, 4), "tokens_per_s": round(pv.B * pv.N / (msv * 1e-3), 1),
                                  "Hq": pv.Hq, "Hkv": pv.Hkv, "query_rho": rho,
                                  "chunk_overlap_16": round(pv.overlap16, 4),
                                  "kernels_avg_ms": {k: round(v["avg_ms"], 4) for k, v in kv.items()}}
        res["extra"]["decode_head_norm"] = bench_decode(torch, hils, synth, WORKLOADS["decode_131k_bf16_b32"],
                                                        args.steps, args.warmup, flags=hils.HILS_FLAG_HEAD_NORM_SELECT)
    if not args.no_cpu:
        res["cpu_baseline"] = cpu_baseline(Wp, host)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
