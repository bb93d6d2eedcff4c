"""The work model behind bench.py's roofline figures, checked against sums written
out row by row (no GPU): the method FLOPs of the chunk pass (QK^T and PV over the
S keys of every selected chunk, 4dS, plus the surrogate score, 2d, per (row,
query head, selected chunk)), of the local pass (4d per window key) and of the
scorers (2d per (head, candidate)), the records the chunk pass writes, and the
decode step's bytes.  Row i's candidates are the chunks that end before its
window starts, C_i = {c : 64 (c + 1) <= i - W + 1} (Sec. 2.1), and its window
the keys from chunk |C_i| on up to i."""
import subprocess
import sys

import bench


def per_row(N, S, W, K):
    rows = []
    for i in range(N):
        nc = max(0, (i - W + 1) // S)
        rows.append((nc, min(K, nc), i - nc * S + 1))
    return rows


def test_prefill_model_matches_row_sums():
    B, Hq, Hkv, N, d, S, K, W = 1, 32, 8, 32768, 128, 64, 16, 512
    rows = per_row(N, S, W, K)
    sel = sum(r[1] for r in rows)
    cand = sum(r[0] for r in rows)
    win = sum(r[2] for r in rows)
    m = bench.prefill_kernel_model(B, Hq, Hkv, N, N, d, S, K, W)
    assert m["k_pf_chunks"]["flop"] == B * Hq * (4 * d * S + 2 * d) * sel
    assert m["k_pf_local"]["flop"] == B * Hq * 4 * d * win
    assert m["k_pf_score"]["flop"] == m["k_pf_sigma"]["flop"] == B * Hq * 2 * d * cand
    assert m["k_pf_select"]["flop"] == 0
    # records: a bf16 d-vector and an fp32 score per (row, query head, selected chunk)
    assert m["k_pf_chunks"]["design_bytes"] == B * Hq * sel * (2 * d + 4)
    # the headline figure quoted in the measurement notes: 536.2 GFLOP per chunk pass
    assert abs(m["k_pf_chunks"]["flop"] / 1e9 - 536.2) < 0.1
    attn, score = bench.prefill_work(B, Hq, Hkv, N, d, S, K, W)
    assert attn == B * Hq * 4 * d * (win + S * sel) and score == B * Hq * 2 * d * cand


def test_decode_bytes_match_the_step():
    # one new token at position ctx of each of 32 sequences: the candidates'
    # landmarks once, the K selected chunks and the window's K/V, q in and out + lse
    B, Hq, Hkv, ctx, d, S, K, W = 32, 32, 8, 131072, 128, 64, 16, 512
    nc = max(0, (ctx - W + 1) // S)
    nloc = ctx - nc * S + 1
    total, parts = bench.decode_bytes(B, Hq, Hkv, Hq, ctx, d, S, K, W)
    assert parts["landmarks"] == B * Hq * nc * d * 2
    assert parts["kv"] == B * Hkv * (min(K, nc) * S + nloc) * d * 2 * 2
    assert parts["q_out"] == B * Hq * d * 2 * 2 + B * Hq * 4
    assert total == sum(parts.values())


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, bench.__file__, "--gpus", "2"], capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "--gpus 2 is not supported" in r.stderr
