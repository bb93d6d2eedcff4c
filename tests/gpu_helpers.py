"""Shared pieces of the GPU parity tests: seeded inputs, the call through the
C-ABI binding, tie-aware selection comparison and the tolerances.

Tolerances (stated once, used by every GPU test):
  * selection: bit-exact, except that a chunk may be swapped for another whose
    group score lies within 1e-4 of the oracle's K-th score (a tie in fp32 vs fp64);
  * f32 outputs: max |d| <= 1e-4;  lse <= 1e-4 (both storage dtypes);
  * bf16 outputs: max |d| <= 2e-2 and mean |d| <= 2e-3;
  * gradients (stored in the input dtype; their magnitudes grow with the number
    of rows that touch a key, up to ~10 here): every element within the max bar
    times max(1, |its reference|) (bf16 storage rounds each element relative to
    its own size), the mean bar times max(1, mean |ref|), and the norm of the
    error within 5e-3 (bf16) / 1e-5 (f32) of the reference's norm.
Outputs are compared with the oracle re-run in forced-index mode on the GPU's
own selection once that selection has been accepted, so a legal tie flip never
shows up as an output error.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
from paper_2607_02980_amd import synth

TIE_TOL = 1e-4
OUT_TOL = {"f32": (1e-4, 1e-4), "bf16": (2e-2, 2e-3)}
LSE_TOL = {"f32": 1e-4, "bf16": 2e-4}


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def oshape(p, N=None) -> oracle.Shape:
    from paper_2607_02980_amd.hils import HILS_FLAG_HEAD_NORM_SELECT

    return oracle.Shape(B=p.B, Hq=p.Hq, Hkv=p.Hkv, Hl=p.Hl or p.Hq, N=p.N if N is None else N, L=p.L, d=p.d,
                        chunk=p.chunk, topk=p.topk, window=p.window,
                        scale=float(np.float32(p.scale if p.scale is not None else p.d ** -0.5)),
                        head_norm=bool(p.flags & HILS_FLAG_HEAD_NORM_SELECT))


def host_inputs(p, wid: int, bias=None, route=False, dout=False, bias_shift=0.0, head_gap=None):
    """Seeded N(0,1) inputs on the host (float32 holding the stored values).

    head_gap = (landmark head, shift): that head's biases are raised by `shift`,
    so its surrogate scores sit far above those of the other heads of its group
    (the per-head fusion must then stabilise every head by its own maximum)."""
    dt = p.dtype
    nc = p.L // p.chunk
    Hl = p.Hl or p.Hq
    t = {
        "q": synth.normal_host((p.B, p.Hq, p.N, p.d), synth.seed_for(wid, "q"), dt),
        "k": synth.normal_host((p.B, p.Hkv, p.L, p.d), synth.seed_for(wid, "k"), dt),
        "v": synth.normal_host((p.B, p.Hkv, p.L, p.d), synth.seed_for(wid, "v"), dt),
        "lmk": synth.normal_host((p.B, Hl, nc, p.d), synth.seed_for(wid, "lmk"), dt),
    }
    if bias or head_gap:
        t["bias"] = synth.normal_host((p.B, Hl, nc), synth.seed_for(wid, "bias"), "f32", std=0.5) + bias_shift
    if head_gap:
        t["bias"][:, head_gap[0], :] += head_gap[1]
    if route:
        t["q_route"] = synth.normal_host((p.B, p.Hq, p.N, p.d), synth.seed_for(wid, "q_route"), dt)
    if dout:
        t["dout"] = synth.normal_host((p.B, p.Hq, p.N, p.d), synth.seed_for(wid, "dout"), dt)
    return t


def to_device(t: dict, p) -> dict:
    out = {}
    for k, v in t.items():
        dt = torch.float32 if k == "bias" else p.torch_dtype
        out[k] = v.to(device="cuda", dtype=dt).contiguous()
    return out


def np32(t):
    return t.detach().float().cpu().numpy() if isinstance(t, torch.Tensor) else t


def check_selection(p, host: dict, gpu_idx: np.ndarray, ref_idx: np.ndarray, qpos=None, rows=None):
    """Tie-aware comparison.  Returns the number of rows that differed (all accepted)."""
    s = oshape(p)
    G = p.Hq // p.Hkv
    diff = 0
    it = rows if rows is not None else [(b, n) for b in range(p.B) for n in range(p.N)]
    for b, n in it:
        for g in range(p.Hkv):
            a, r = gpu_idx[b, g, n], ref_idx[b, g, n]
            if np.array_equal(a, r):
                continue
            diff += 1
            sig = oracle.group_scores(s, np32(host["q"]), np32(host["lmk"]), b, g, n,
                                      bias=np32(host.get("bias")), q_route=np32(host.get("q_route")), qpos=qpos)
            sel_r = set(int(c) for c in r if c >= 0)
            sel_a = set(int(c) for c in a if c >= 0)
            assert len(sel_a) == len(sel_r), f"row (b={b}, g={g}, n={n}): {len(sel_a)} vs {len(sel_r)} chunks"
            assert list(a[: len(sel_a)]) == sorted(sel_a) and all(a[len(sel_a):] == -1), f"row {b, g, n} layout {a}"
            kth = min(sig[c] for c in sel_r)
            for c in sel_a ^ sel_r:
                assert abs(sig[c] - kth) <= TIE_TOL, (
                    f"row (b={b}, g={g}, n={n}): chunk {c} score {sig[c]:.6f} vs K-th {kth:.6f}; gpu {a} ref {r}")
    return diff


REL_NORM_TOL = {"f32": 1e-5, "bf16": 5e-3}


def check_close(name, got, ref, dtype, rel=False):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{name}: non-finite values"
    d = np.abs(got - ref)
    mx_tol, mean_tol = OUT_TOL[dtype]
    rel_err = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    if rel:
        # gradients: each element against its own magnitude
        scale = np.maximum(1.0, np.abs(ref))
        worst = float((d / scale).max())
        mean_tol *= max(1.0, float(np.abs(ref).mean()))
        log(f"  {name}: max|d|={d.max():.3e} max|d|/max(1,|ref|)={worst:.3e} (tol {mx_tol:.1e}) "
            f"mean|d|={d.mean():.3e} (tol {mean_tol:.1e}) rel={rel_err:.2e} (tol {REL_NORM_TOL[dtype]:.0e})")
        assert worst <= mx_tol, f"{name}: an element's |d| / max(1, |ref|) is {worst:.3e} > {mx_tol:.1e}"
        assert rel_err <= REL_NORM_TOL[dtype], f"{name}: |d| / |ref| = {rel_err:.2e}"
    else:
        log(f"  {name}: max|d|={d.max():.3e} (tol {mx_tol:.1e}) mean|d|={d.mean():.3e} (tol {mean_tol:.1e}) "
            f"rel={rel_err:.2e}")
        assert d.max() <= mx_tol, f"{name}: max |d| {d.max():.3e} > {mx_tol:.1e}"
    assert d.mean() <= mean_tol, f"{name}: mean |d| {d.mean():.3e} > {mean_tol:.1e}"


def check_lse(got, ref, dtype):
    d = np.abs(np.asarray(got, np.float64) - np.asarray(ref, np.float64))
    log(f"  lse: max|d|={d.max():.3e} (tol {LSE_TOL[dtype]:.0e})")
    assert d.max() <= LSE_TOL[dtype]
