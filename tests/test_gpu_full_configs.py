"""GPU parity at the full workload sizes, in the launch configuration bench.py
times, on outputs the oracle computes one by one.

* 32K prefill (bf16): selection and outputs of ~600 sampled query rows (edges
  of the window, chunk boundaries, first/last rows, seeded random rows), and
  for every row the properties that hold at any size: idx ascending, -1 only
  as padding, exactly min(K, |C_i|) chunks, all in C_i; out and lse finite.
* 131K decode (32 sequences) and 1M decode (4 sequences): the selection and
  the outputs of every sequence and KV group.  The oracle gets
  sparse host copies of the caches holding exactly the positions the row can
  attend with the checked selection (local window + the selected chunks), so
  only those slices leave the GPU.
* 16K x 4 training shape: forward rows, dq of sampled rows, and dk/dv/dk'/db'
  of sampled chunks, for which the oracle runs exactly the rows that touch the
  chunk (its local-window rows and the rows that selected it).
Inputs are drawn exactly as bench.py draws them.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_02980_amd import synth
from paper_2607_02980_amd.configs import WORKLOADS
from tests.gpu_helpers import check_close, check_lse, check_selection, log, np32, oshape

pytestmark = pytest.mark.gpu


def params_of(W, hils):
    return hils.Params(B=W.B, Hq=W.Hq, Hkv=W.Hkv, N=W.N, L=W.L, d=W.d, chunk=W.chunk, topk=W.topk,
                       window=W.window, dtype=W.dtype)


def n_cand(i, S, Wn):
    return max(0, (i - Wn + 1) // S)


def sampled_rows(N, W, extra, seed):
    special = [0, 1, 63, 64, W - 2, W - 1, W, W + 63, W + 64, 1000, N // 2, N - 65, N - 64, N - 2, N - 1]
    rng = np.random.default_rng(seed)
    rnd = rng.integers(0, N, extra).tolist()
    return sorted(set(n for n in special + rnd if 0 <= n < N))


def test_prefill_32k_bf16_sampled_rows():
    from paper_2607_02980_amd import hils

    W = WORKLOADS["prefill_32k_bf16"]
    p = params_of(W, hils)
    log(f"[full] {W.name}: generating inputs")
    nc = p.L // p.chunk
    host = {
        "q": synth.normal_host((p.B, p.Hq, p.N, p.d), synth.seed_for(W.wid, "q"), p.dtype),
        "k": synth.normal_host((p.B, p.Hkv, p.L, p.d), synth.seed_for(W.wid, "k"), p.dtype),
        "v": synth.normal_host((p.B, p.Hkv, p.L, p.d), synth.seed_for(W.wid, "v"), p.dtype),
        "lmk": synth.normal_host((p.B, p.Hq, nc, p.d), synth.seed_for(W.wid, "lmk"), p.dtype),
    }
    dev = {k: v.to("cuda", torch.bfloat16).contiguous() for k, v in host.items()}
    log(f"[full] {W.name}: GPU prefill")
    out, lse, idx = hils.hils_prefill_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"])
    torch.cuda.synchronize()
    gidx = idx.cpu().numpy()
    assert (gidx >= -1).all() and (gidx < nc).all()
    # every row: the selection's shape (ascending, padded, min(K, |C_i|) chunks of C_i)
    ncand = np.maximum(0, (np.arange(p.N) - p.window + 1) // p.chunk)
    valid = gidx >= 0
    assert (valid.sum(-1) == np.minimum(p.topk, ncand)[None, None, :]).all(), "selection sizes"
    assert (valid[..., 1:] <= valid[..., :-1]).all(), "-1 only as trailing padding"
    steps = np.diff(gidx.astype(np.int64), axis=-1)
    assert (steps[valid[..., 1:]] > 0).all(), "valid entries strictly ascending"
    assert (np.where(valid, gidx, -1) < ncand[None, None, :, None]).all(), "chunks in C_i"
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all(), "finite outputs"
    log(f"  all {p.N * p.Hkv} selection rows: sizes, order and range hold")
    rows_n = sampled_rows(p.N, p.window, 600, 2)
    rows = np.array([(0, n) for n in rows_n], np.int32)
    s = oshape(p)
    arr = {k: v.numpy() for k, v in host.items()}
    log(f"[full] {W.name}: oracle on {len(rows)} rows")
    ref = oracle.fwd(s, arr["q"], arr["k"], arr["v"], arr["lmk"], rows=rows)
    nd = check_selection(p, host, gidx, ref["idx"], rows=[tuple(r) for r in rows])
    log(f"  selection: {nd} rows differ only by accepted ties")
    ref = oracle.fwd(s, arr["q"], arr["k"], arr["v"], arr["lmk"], rows=rows, idx=gidx)
    o, l = np32(out), np32(lse)
    check_close("out(sampled rows)", o[0][:, rows_n], ref["out"][0][:, rows_n], p.dtype)
    check_lse(l[0][:, rows_n], ref["lse"][0][:, rows_n], p.dtype)


LONG_CASES = {
    # name: (N = L, Hq, Hkv, flags, extra rows).  40K tokens: 625 candidate chunks,
    # the split scorer with 16 registers of candidates per lane; 66,560 tokens: 1,040
    # chunks, beyond the split scorer, so the fused one with five 256-candidate slices
    # per row (every prefill beyond 64K tokens takes it); each under the raw and the
    # per-head normalised ranking (the log-sum-exp pass first)
    "split_625_chunks": (40000, 8, 2, 0, [33280, 33343, 33344, 36000]),
    "split_625_chunks_head_norm": (40000, 8, 2, 4, [33280, 33343, 33344, 36000]),
    "fused_1040_chunks": (66560, 4, 1, 0, [65600, 66111, 66112, 66500]),
    "fused_1040_chunks_head_norm": (66560, 4, 1, 4, [65600, 66111, 66112, 66500]),
}


@pytest.mark.parametrize("name", list(LONG_CASES))
def test_prefill_long_sequence_scorers(name):
    from paper_2607_02980_amd import hils

    N, Hq, Hkv, flags, extra = LONG_CASES[name]
    p = hils.Params(B=1, Hq=Hq, Hkv=Hkv, N=N, L=N, d=64, topk=16, window=512, dtype="bf16", flags=flags)
    nc = p.L // p.chunk
    wid = 31
    host = {
        "q": synth.normal_host((p.B, p.Hq, p.N, p.d), synth.seed_for(wid, "q"), p.dtype),
        "k": synth.normal_host((p.B, p.Hkv, p.L, p.d), synth.seed_for(wid, "k"), p.dtype),
        "v": synth.normal_host((p.B, p.Hkv, p.L, p.d), synth.seed_for(wid, "v"), p.dtype),
        "lmk": synth.normal_host((p.B, p.Hq, nc, p.d), synth.seed_for(wid, "lmk"), p.dtype),
    }
    dev = {k: v.to("cuda", torch.bfloat16).contiguous() for k, v in host.items()}
    log(f"[long] case={name} N=L={p.N} ({nc} chunks) flags={flags}: GPU prefill")
    out, lse, idx = hils.hils_prefill_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"])
    torch.cuda.synchronize()
    gidx = idx.cpu().numpy()
    ncand = np.maximum(0, (np.arange(p.N) - p.window + 1) // p.chunk)
    valid = gidx >= 0
    assert (valid.sum(-1) == np.minimum(p.topk, ncand)[None, None, :]).all(), "selection sizes"
    assert (valid[..., 1:] <= valid[..., :-1]).all(), "-1 only as trailing padding"
    steps = np.diff(gidx.astype(np.int64), axis=-1)
    assert (steps[valid[..., 1:]] > 0).all(), "valid entries strictly ascending"
    assert (np.where(valid, gidx, -1) < ncand[None, None, :, None]).all(), "chunks in C_i"
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all(), "finite outputs"
    rows_n = sorted(set(sampled_rows(p.N, p.window, 120, 7) + extra))
    rows = np.array([(0, n) for n in rows_n], np.int32)
    s = oshape(p)
    arr = {k: v.numpy() for k, v in host.items()}
    log(f"  oracle on {len(rows)} rows")
    ref = oracle.fwd(s, arr["q"], arr["k"], arr["v"], arr["lmk"], rows=rows)
    nd = check_selection(p, host, gidx, ref["idx"], rows=[tuple(r) for r in rows])
    log(f"  selection: {nd} rows differ only by accepted ties")
    ref = oracle.fwd(s, arr["q"], arr["k"], arr["v"], arr["lmk"], rows=rows, idx=gidx)
    o, l = np32(out), np32(lse)
    check_close("out(sampled rows)", o[0][:, rows_n], ref["out"][0][:, rows_n], p.dtype)
    check_lse(l[0][:, rows_n], ref["lse"][0][:, rows_n], p.dtype)


def _decode_device_inputs(W, p):
    nc = p.L // p.chunk
    return {
        "q": synth.normal_device((p.B, p.Hq, 1, p.d), synth.seed_for(W.wid, "q"), p.dtype, "cuda"),
        "k": synth.normal_device((p.B, p.Hkv, p.L, p.d), synth.seed_for(W.wid, "k"), p.dtype, "cuda"),
        "v": synth.normal_device((p.B, p.Hkv, p.L, p.d), synth.seed_for(W.wid, "v"), p.dtype, "cuda"),
        "lmk": synth.normal_device((p.B, p.Hq, nc, p.d), synth.seed_for(W.wid, "lmk"), p.dtype, "cuda"),
    }


def _sparse_kv(dev, b, p, pos, sel_by_group):
    """Host float32 copies of sequence b's caches that hold only what row `pos`
    attends: the local window and, per KV group, its selected chunks."""
    S = p.chunk
    k = np.zeros((1, p.Hkv, p.L, p.d), np.float32)
    v = np.zeros((1, p.Hkv, p.L, p.d), np.float32)
    ell = n_cand(pos, S, p.window) * S
    k[0, :, ell:pos + 1] = np32(dev["k"][b, :, ell:pos + 1])
    v[0, :, ell:pos + 1] = np32(dev["v"][b, :, ell:pos + 1])
    for g, chunks in enumerate(sel_by_group):
        for c in chunks:
            k[0, g, c * S:(c + 1) * S] = np32(dev["k"][b, g, c * S:(c + 1) * S])
            v[0, g, c * S:(c + 1) * S] = np32(dev["v"][b, g, c * S:(c + 1) * S])
    return k, v


def _run_decode_full(name, check_out):
    from paper_2607_02980_amd import hils

    W = WORKLOADS[name]
    p = hils.Params(B=W.B, Hq=W.Hq, Hkv=W.Hkv, N=1, L=W.L, d=W.d, chunk=W.chunk, topk=W.topk, window=W.window,
                    dtype=W.dtype)
    log(f"[full] {name}: generating caches on the device")
    dev = _decode_device_inputs(W, p)
    seqlens = torch.full((p.B,), W.ctx + 1, dtype=torch.int32, device="cuda")
    log(f"[full] {name}: GPU decode")
    out, lse, idx = hils.hils_decode_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"], seqlens=seqlens)
    torch.cuda.synchronize()
    gidx = idx.cpu().numpy()
    pos = W.ctx
    q_h = np32(dev["q"])
    p1 = hils.Params(**{**p.__dict__, "B": 1})
    s1 = oshape(p1)
    qpos = np.array([[pos]], np.int32)
    for b in range(p.B):
        lmk_b = np32(dev["lmk"][b:b + 1])
        host_b = {"q": q_h[b:b + 1], "lmk": lmk_b}
        zk = np.zeros((1, p.Hkv, p.L, p.d), np.float32)
        ref = oracle.fwd(s1, q_h[b:b + 1], zk, zk, lmk_b, qpos=qpos)  # selection only
        nd = check_selection(p1, host_b, gidx[b:b + 1], ref["idx"], qpos=qpos)
        if b in check_out:
            sel = [[int(c) for c in gidx[b, g, 0] if c >= 0] for g in range(p.Hkv)]
            k, v = _sparse_kv(dev, b, p, pos, sel)
            r2 = oracle.fwd(s1, q_h[b:b + 1], k, v, lmk_b, qpos=qpos, idx=gidx[b:b + 1])
            log(f"  sequence {b}: selection ok ({nd} tie rows); outputs:")
            check_close("out", np32(out[b:b + 1]), r2["out"], p.dtype)
            check_lse(np32(lse[b:b + 1]), r2["lse"], p.dtype)
    del dev
    torch.cuda.empty_cache()


def test_decode_131k_bf16_b32_all_sequences():
    _run_decode_full("decode_131k_bf16_b32", check_out=set(range(32)))


def test_decode_1m_bf16_b4_all_sequences():
    _run_decode_full("decode_1m_bf16_b4", check_out=set(range(4)))


def test_train_16k_bf16_b4_sampled():
    from paper_2607_02980_amd import hils

    W = WORKLOADS["train_16k_bf16_b4"]
    p = params_of(W, hils)
    nc = p.L // p.chunk
    log(f"[full] {W.name}: generating inputs on the device")
    dev = {
        "q": synth.normal_device((p.B, p.Hq, p.N, p.d), synth.seed_for(W.wid, "q"), p.dtype, "cuda"),
        "k": synth.normal_device((p.B, p.Hkv, p.L, p.d), synth.seed_for(W.wid, "k"), p.dtype, "cuda"),
        "v": synth.normal_device((p.B, p.Hkv, p.L, p.d), synth.seed_for(W.wid, "v"), p.dtype, "cuda"),
        "lmk": synth.normal_device((p.B, p.Hq, nc, p.d), synth.seed_for(W.wid, "lmk"), p.dtype, "cuda"),
        "dout": synth.normal_device((p.B, p.Hq, p.N, p.d), synth.seed_for(W.wid, "dout"), p.dtype, "cuda"),
    }
    log(f"[full] {W.name}: GPU forward + backward")
    out, lse, idx = hils.hils_prefill_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"])
    g = hils.hils_bwd(p, dev["dout"], dev["q"], dev["k"], dev["v"], dev["lmk"], out, lse, idx)
    torch.cuda.synchronize()
    host = {k: np32(v) for k, v in dev.items()}
    gidx = idx.cpu().numpy()
    s = oshape(p)
    rng = np.random.default_rng(5)
    rows = [(b, n) for b in range(p.B) for n in sampled_rows(p.N, p.window, 40, 50 + b)]
    rows_a = np.array(rows, np.int32)
    log(f"[full] {W.name}: oracle forward on {len(rows)} rows")
    ref = oracle.fwd(s, host["q"], host["k"], host["v"], host["lmk"], rows=rows_a)
    nd = check_selection(p, {"q": host["q"], "lmk": host["lmk"]}, gidx, ref["idx"], rows=rows)
    log(f"  selection: {nd} rows differ only by accepted ties")
    ref = oracle.fwd(s, host["q"], host["k"], host["v"], host["lmk"], rows=rows_a, idx=gidx)
    o, l = np32(out), np32(lse)
    bi, ni = rows_a[:, 0], rows_a[:, 1]
    check_close("out(sampled rows)", o[bi, :, ni], ref["out"][bi, :, ni], p.dtype)
    check_lse(l[bi, :, ni], ref["lse"][bi, :, ni], p.dtype)

    log(f"[full] {W.name}: oracle dq on {len(rows)} rows")
    rb = oracle.bwd(s, host["dout"], host["q"], host["k"], host["v"], host["lmk"], gidx, rows=rows_a)
    check_close("dq(sampled rows)", np32(g["dq"])[bi, :, ni], rb["dq"][bi, :, ni], p.dtype, rel=True)
    del rb

    G = p.Hq // p.Hkv
    # chunk 5 is retrieved by rows spread over more than one 8192-row window of the list sort
    for (b, gg, c) in [(0, 0, 5), (1, 3, 200), (3, 6, 240), (2, 1, 64), (0, 7, 130)]:
        lo, hi = c * p.chunk, min(p.N - 1, (c + 1) * p.chunk + p.window - 2)
        local = list(range(lo, hi + 1))
        picked = [n for n in range(p.N) if c in gidx[b, gg, n]]
        rr = np.array([(b, n) for n in sorted(set(local + picked))], np.int32)
        log(f"[full] {W.name}: oracle dk/dv/dlmk for chunk (b={b}, g={gg}, c={c}): {len(rr)} rows "
            f"({len(picked)} retrievals)")
        rb = oracle.bwd(s, host["dout"], host["q"], host["k"], host["v"], host["lmk"], gidx, rows=rr,
                        only_group=gg)
        sl = slice(c * p.chunk, (c + 1) * p.chunk)
        check_close("dk(chunk)", np32(g["dk"])[b, gg, sl], rb["dk"][b, gg, sl], p.dtype, rel=True)
        check_close("dv(chunk)", np32(g["dv"])[b, gg, sl], rb["dv"][b, gg, sl], p.dtype, rel=True)
        hs = slice(gg * G, (gg + 1) * G)
        check_close("dlmk(chunk)", np32(g["dlmk"])[b, hs, c], rb["dlmk"][b, hs, c], p.dtype, rel=True)
        check_close("dlmk_bias(chunk)", np32(g["dlmk_bias"])[b, hs, c], rb["dbias"][b, hs, c], p.dtype, rel=True)
    log(f"[full] {W.name}: backward repeated, bitwise equal")
    g2 = hils.hils_bwd(p, dev["dout"], dev["q"], dev["k"], dev["v"], dev["lmk"], out, lse, idx)
    torch.cuda.synchronize()
    for key in g:
        if g[key] is not None:
            assert torch.equal(g[key], g2[key]), key
    del dev, g, g2
    torch.cuda.empty_cache()
