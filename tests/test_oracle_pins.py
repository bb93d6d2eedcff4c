"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these re-types the oracle's arithmetic: each compares it with an
independent statement -- a hand-derived worked example, textbook dense causal
attention, naive block-sparse attention, brute-force subset search, the
paper's second (dense, case-wise) formulation, finite differences, or torch
autograd of dense attention -- under constructions where HiLS must equal them.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle
from tests.oracle_helpers import (brute_force_topk, dense_causal, group_scores_np, naive_bsa, p1_landmarks,
                                  p2_construction)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_worked_example.txt")


def rnd(rng, *shape):
    return rng.standard_normal(shape).astype(np.float32)


# ---------------------------------------------------------------- golden ---

def _parse_value(tok):
    if tok.startswith("log"):
        return math.log(float(tok[3:]))
    if "/" in tok:
        a, b = tok.split("/")
        return float(a) / float(b)
    return float(tok)


def test_hand_worked_example():
    """Sec. 2.1, Eqs. (1), (9), (10) and App. C worked by hand on a 6-token toy."""
    rows = [ln.split() for ln in open(GOLDEN) if ln.strip() and not ln.startswith("#")]
    ln3, ln5 = math.log(3.0), math.log(5.0)
    for case in ("A", "B"):
        Hq = 1 if case == "A" else 2
        s = oracle.Shape(B=1, Hq=Hq, Hkv=1, Hl=Hq, N=6, L=6, d=1, chunk=2, topk=1, window=1, scale=1.0)
        q = np.ones((1, Hq, 6, 1), np.float32)
        k = np.zeros((1, 1, 6, 1), np.float32)
        v = np.arange(6, dtype=np.float32).reshape(1, 1, 6, 1)
        # L/S = 3 landmark rows; the third (chunk 2) is never a candidate here
        if case == "A":
            lmk = np.array([0.0, ln3, 9.0], np.float32).reshape(1, 1, 3, 1)
        else:
            lmk = np.array([[0.0, ln3, 9.0], [ln5, 0.0, 9.0]], np.float32).reshape(1, 2, 3, 1)
        r = oracle.fwd(s, q, k, v, lmk)
        for c, head, i, idx0, out, lse in rows:
            if c != case:
                continue
            head, i, idx0 = int(head), int(i), int(idx0)
            assert r["idx"][0, 0, i, 0] == idx0, (case, head, i)
            # landmarks are float32-rounded logs: 1e-7 slack
            assert abs(r["out"][0, head, i, 0] - _parse_value(out)) < 1e-6, (case, head, i)
            assert abs(r["lse"][0, head, i] - _parse_value(lse)) < 1e-6, (case, head, i)


# ------------------------------------------------- reductions to dense ---

@pytest.mark.parametrize("Hq,Hkv,Hl", [(1, 1, 1), (4, 1, 4), (4, 2, 2), (6, 2, 6)])
def test_p1_chunk1_window1_topall_is_dense_causal(Hq, Hkv, Hl):
    """P1: S=1, W=1, k'_c = k_c, no bias, K >= N  =>  dense causal attention."""
    rng = np.random.default_rng(11)
    B, N, d = 2, 37, 8
    q, k, v = rnd(rng, B, Hq, N, d), rnd(rng, B, Hkv, N, d), rnd(rng, B, Hkv, N, d)
    lmk = p1_landmarks(k, Hq, Hl)
    s = oracle.Shape(B=B, Hq=Hq, Hkv=Hkv, Hl=Hl, N=N, L=N, d=d, chunk=1, topk=N, window=1, scale=0.3)
    r = oracle.fwd(s, q, k, v, lmk)
    ref, ref_lse = dense_causal(q, k, v, 0.3)
    np.testing.assert_allclose(r["out"], ref, atol=1e-12, rtol=0)
    np.testing.assert_allclose(r["lse"], ref_lse, atol=1e-12, rtol=0)


@pytest.mark.parametrize("S,W,N", [(4, 1, 48), (4, 5, 50), (8, 8, 64), (8, 9, 61), (16, 24, 128), (2, 3, 33)])
@pytest.mark.parametrize("Hq,Hkv,Hl", [(2, 1, 2), (4, 2, 2)])
def test_p2_exact_mass_landmarks_top_all_is_dense_causal(S, W, N, Hq, Hkv, Hl):
    """P2: constant keys inside each chunk, k'_c = kappa_c, b'_c = log S  =>
    s^_c = log Z_c exactly, and with K >= |C_i| HiLS is dense causal attention."""
    rng = np.random.default_rng(S * 100 + W)
    B, d = 1, 8
    L = -(-N // S) * S
    kappa, k, lmk, bias = p2_construction(rng, B, Hq, Hkv, Hl, L, d, S)
    q, v = rnd(rng, B, Hq, N, d), rnd(rng, B, Hkv, L, d)
    s = oracle.Shape(B=B, Hq=Hq, Hkv=Hkv, Hl=Hl, N=N, L=L, d=d, chunk=S, topk=L // S, window=W, scale=0.5)
    r = oracle.fwd(s, q, k, v, lmk, bias=bias)
    ref, ref_lse = dense_causal(q, k, v, 0.5)
    # bias log S is float32-rounded: relative 1e-7 in the chunk weights
    np.testing.assert_allclose(r["out"], ref, atol=2e-7, rtol=0)
    np.testing.assert_allclose(r["lse"], ref_lse, atol=2e-7, rtol=0)


@pytest.mark.parametrize("S,W,N", [(4, 64, 60), (8, 1, 8), (16, 16, 16)])
def test_p3_no_candidates_is_dense_causal(S, W, N):
    """P3: N <= W, or N <= S with W = 1  =>  C_i is empty for every query."""
    rng = np.random.default_rng(3)
    B, Hq, Hkv, d = 1, 4, 2, 16
    L = -(-N // S) * S
    q, k, v = rnd(rng, B, Hq, N, d), rnd(rng, B, Hkv, L, d), rnd(rng, B, Hkv, L, d)
    lmk = rnd(rng, B, Hq, L // S, d)
    s = oracle.Shape(B=B, Hq=Hq, Hkv=Hkv, Hl=Hq, N=N, L=L, d=d, chunk=S, topk=3, window=W, scale=0.25)
    r = oracle.fwd(s, q, k, v, lmk)
    ref, ref_lse = dense_causal(q, k, v, 0.25)
    np.testing.assert_allclose(r["out"], ref, atol=1e-12)
    np.testing.assert_allclose(r["lse"], ref_lse, atol=1e-12)
    assert (r["idx"] == -1).all()


def test_p9_equals_naive_bsa_with_exact_mass_landmarks():
    """P9: with the P2 construction and G = 1, HiLS (K < |C_i|) selects the same
    chunks as naive BSA (Eq. (2)) and produces the same weights (Eq. (3))."""
    rng = np.random.default_rng(9)
    B, H, N, d, S, W, K = 1, 2, 96, 8, 4, 6, 3
    kappa, k, lmk, bias = p2_construction(rng, B, H, H, H, N, d, S)
    q, v = rnd(rng, B, H, N, d), rnd(rng, B, H, N, d)
    s = oracle.Shape(B=B, Hq=H, Hkv=H, Hl=H, N=N, L=N, d=d, chunk=S, topk=K, window=W, scale=0.7)
    r = oracle.fwd(s, q, k, v, lmk, bias=bias)
    ref, ref_idx = naive_bsa(q, k, v, 0.7, S, W, K)
    assert (r["idx"] == ref_idx).all()
    np.testing.assert_allclose(r["out"], ref, atol=2e-7)


# ------------------------------------------------------------ selection ---

@pytest.mark.parametrize("Hq,Hkv,Hl,route,with_bias", [(1, 1, 1, False, False), (4, 1, 4, False, True),
                                                        (4, 2, 2, True, True), (4, 1, 1, True, False)])
def test_p5_selection_is_brute_force_maximiser(Hq, Hkv, Hl, route, with_bias):
    """P5: I_i maximises the sum of group scores over all K-subsets of C_i
    (Eq. (9) with App. C's max over heads), checked by exhaustive search."""
    rng = np.random.default_rng(5 + Hq + Hl)
    B, N, d, S, W, K = 1, 44, 8, 4, 5, 3
    q, k, v = rnd(rng, B, Hq, N, d), rnd(rng, B, Hkv, N, d), rnd(rng, B, Hkv, N, d)
    lmk = rnd(rng, B, Hl, N // S, d)
    bias = rnd(rng, B, Hl, N // S) if with_bias else None
    qr = rnd(rng, B, Hq, N, d) if route else None
    s = oracle.Shape(B=B, Hq=Hq, Hkv=Hkv, Hl=Hl, N=N, L=N, d=d, chunk=S, topk=K, window=W, scale=0.4)
    r = oracle.fwd(s, q, k, v, lmk, bias=bias, q_route=qr)
    G = Hq // Hkv
    for g in range(Hkv):
        for n in range(N):
            nc = oracle.n_candidates(n, S, W)
            sig = group_scores_np(qr if route else q, lmk, bias, 0.4, 0, g, n, n, G, Hl, Hq, nc)
            np.testing.assert_allclose(oracle.group_scores(s, q, lmk, 0, g, n, bias=bias, q_route=qr), sig,
                                       atol=1e-12)
            best = brute_force_topk(sig, K)
            assert len(best) == 1
            got = [c for c in r["idx"][0, g, n] if c >= 0]
            assert tuple(got) == best[0], (g, n)
            assert list(r["idx"][0, g, n, len(got):]) == [-1] * (K - len(got))


def test_ties_go_to_the_smaller_chunk_index():
    """Reading of rank_desc ties (Eq. (9)): equal group scores prefer the smaller c."""
    B, Hq, Hkv, N, d, S, W, K = 1, 2, 1, 40, 4, 4, 1, 2
    rng = np.random.default_rng(1)
    q = np.ones((B, Hq, N, d), np.float32)
    k, v = rnd(rng, B, Hkv, N, d), rnd(rng, B, Hkv, N, d)
    nc = N // S
    lmk = np.zeros((B, Hq, nc, d), np.float32)
    lmk[0, 0, [2, 5, 7], :] = 1.0  # head 0 ties on three chunks
    lmk[0, 1, [1, 6], :] = 1.0     # head 1 ties with them on two more
    s = oracle.Shape(B=B, Hq=Hq, Hkv=Hkv, Hl=Hq, N=N, L=N, d=d, chunk=S, topk=K, window=W, scale=1.0)
    r = oracle.fwd(s, q, k, v, lmk)
    assert list(r["idx"][0, 0, 39]) == [1, 2]   # five-way tie -> the two smallest
    assert list(r["idx"][0, 0, 8]) == [0, 1]    # C = {0, 1}: chunk 1 top, then chunk 0
    assert list(r["idx"][0, 0, 4]) == [0, -1]   # |C| = 1 < K: padded


# ------------------------------------------------------------ invariants ---

def test_p4_invariants_and_p6_dense_form():
    """P4: fusion weights are a distribution, lse >= log Z_swa, outputs lie in
    the hull of the attended values.  P6: the factored forward equals the dense
    case-wise weights of App. C applied to V, and those rows sum to one."""
    rng = np.random.default_rng(4)
    B, Hq, Hkv, N, d, S, W, K = 2, 4, 2, 70, 8, 4, 7, 3
    q, k, v = rnd(rng, B, Hq, N, d), rnd(rng, B, Hkv, 72, d), rnd(rng, B, Hkv, 72, d)
    lmk, bias, qr = rnd(rng, B, Hq, 18, d), rnd(rng, B, Hq, 18), rnd(rng, B, Hq, N, d)
    s = oracle.Shape(B=B, Hq=Hq, Hkv=Hkv, Hl=Hq, N=N, L=72, d=d, chunk=S, topk=K, window=W, scale=0.35)
    r = oracle.fwd(s, q, k, v, lmk, bias=bias, q_route=qr, want_debug=True)
    a = r["alpha"]
    assert (a >= 0).all()
    np.testing.assert_allclose(a.sum(-1), 1.0, atol=1e-12)
    assert (r["lse"] >= np.log(a[..., 0]) + r["lse"] - 1e-12).all()  # alpha0 <= 1
    w = oracle.dense_weights(s, q, k, lmk, r["idx"], bias=bias, q_route=qr)
    np.testing.assert_allclose(w.sum(-1), 1.0, atol=1e-12)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            dense_out = w[b, h] @ v[b, h // G].astype(np.float64)
            np.testing.assert_allclose(r["out"][b, h], dense_out, atol=1e-12)
            for n in range(N):
                att = np.nonzero(w[b, h, n])[0]
                vv = v[b, h // G, att].astype(np.float64)
                assert (r["out"][b, h, n] <= vv.max(0) + 1e-12).all()
                assert (r["out"][b, h, n] >= vv.min(0) - 1e-12).all()


def test_f32_oracle_agrees_with_f64():
    rng = np.random.default_rng(2)
    B, Hq, Hkv, N, d, S, W, K = 1, 4, 1, 256, 32, 16, 40, 4
    q, k, v = rnd(rng, B, Hq, N, d), rnd(rng, B, Hkv, N, d), rnd(rng, B, Hkv, N, d)
    lmk = rnd(rng, B, Hq, N // S, d)
    s = oracle.Shape(B=B, Hq=Hq, Hkv=Hkv, Hl=Hq, N=N, L=N, d=d, chunk=S, topk=K, window=W, scale=d ** -0.5)
    r64 = oracle.fwd(s, q, k, v, lmk)
    r32 = oracle.fwd(s, q, k, v, lmk, prec="f32")
    assert (r64["idx"] == r32["idx"]).all()
    np.testing.assert_allclose(r32["out"], r64["out"], atol=1e-5)


def test_forced_index_validation():
    rng = np.random.default_rng(0)
    s = oracle.Shape(B=1, Hq=1, Hkv=1, Hl=1, N=16, L=16, d=4, chunk=4, topk=2, window=1, scale=1.0)
    q, k, v, lmk = rnd(rng, 1, 1, 16, 4), rnd(rng, 1, 1, 16, 4), rnd(rng, 1, 1, 16, 4), rnd(rng, 1, 1, 4, 4)
    idx = np.full((1, 1, 16, 2), -1, np.int32)
    idx[0, 0, 5] = [1, -1]  # chunk 1 is not a candidate of query 5 (C = {0})
    with pytest.raises(ValueError):
        oracle.fwd(s, q, k, v, lmk, idx=idx)
    idx[0, 0, 5] = [0, -1]
    idx[0, 0, 15] = [2, 1]  # not ascending
    with pytest.raises(ValueError):
        oracle.fwd(s, q, k, v, lmk, idx=idx)


# --------------------------------------------------------------- backward ---

def _quantised(rng, *shape):
    # multiples of 2^-6 in [-2, 2]: x +- 2^-14 stays exact in float32
    return np.clip(np.round(rng.standard_normal(shape) * 64) / 64, -2, 2).astype(np.float32)


@pytest.mark.parametrize("Hl_is_Hq,route,with_bias", [(True, True, True), (False, False, True), (True, False, False)])
def test_p7_backward_matches_finite_differences(Hl_is_Hq, route, with_bias):
    """P7: central differences of the fp64 forward (selection held fixed) equal
    every gradient of the backward: dq, dk, dv, dk', db' and dq^."""
    rng = np.random.default_rng(7)
    B, Hq, Hkv, N, d, S, W, K = 1, 4, 2, 11, 3, 2, 3, 2
    L = 12
    Hl = Hq if Hl_is_Hq else Hkv
    T = {"q": _quantised(rng, B, Hq, N, d), "k": _quantised(rng, B, Hkv, L, d), "v": _quantised(rng, B, Hkv, L, d),
         "lmk": _quantised(rng, B, Hl, L // S, d)}
    if with_bias:
        T["bias"] = _quantised(rng, B, Hl, L // S)
    if route:
        T["q_route"] = _quantised(rng, B, Hq, N, d)
    s = oracle.Shape(B=B, Hq=Hq, Hkv=Hkv, Hl=Hl, N=N, L=L, d=d, chunk=S, topk=K, window=W, scale=0.5)
    dout = _quantised(rng, B, Hq, N, d).astype(np.float64)
    base = oracle.fwd(s, **T)
    idx = base["idx"]

    def loss(TT):
        return float((oracle.fwd(s, idx=idx, **TT)["out"] * dout).sum())

    g = oracle.bwd(s, dout.astype(np.float32), idx=idx, **T)
    names = {"q": "dq", "k": "dk", "v": "dv", "lmk": "dlmk", "bias": "dbias", "q_route": "dq_route"}
    h = 2.0 ** -14
    for name, arr in T.items():
        fd = np.zeros(arr.shape)
        for pos in np.ndindex(arr.shape):
            TT = dict(T)
            a = arr.copy()
            a[pos] = arr[pos] + h
            TT[name] = a
            fp = loss(TT)
            a = arr.copy()
            a[pos] = arr[pos] - h
            TT[name] = a
            fm = loss(TT)
            fd[pos] = (fp - fm) / (2 * h)
        np.testing.assert_allclose(g[names[name]], fd, atol=2e-7, rtol=1e-6, err_msg=name)


def _torch_dense_grads(q, k, v, dout, scale):
    qt = torch.tensor(q, dtype=torch.float64, requires_grad=True)
    kt = torch.tensor(k, dtype=torch.float64, requires_grad=True)
    vt = torch.tensor(v, dtype=torch.float64, requires_grad=True)
    G = q.shape[1] // k.shape[1]
    kk = kt.repeat_interleave(G, dim=1)
    vv = vt.repeat_interleave(G, dim=1)
    N, L = q.shape[2], k.shape[2]
    s = scale * qt @ kk.transpose(-1, -2)
    mask = torch.arange(L)[None, :] > torch.arange(N)[:, None]
    s = s.masked_fill(mask, float("-inf"))
    out = torch.softmax(s, -1) @ vv
    (out * torch.tensor(dout)).sum().backward()
    return qt.grad.numpy(), kt.grad.numpy(), vt.grad.numpy()


def test_p7_backward_reduces_to_dense_attention_gradients():
    """P7 under P1: gradients equal torch autograd of dense causal attention;
    the key gradient splits into the token path (dk) and the landmark path
    (dk' summed over the group's landmark heads)."""
    rng = np.random.default_rng(17)
    B, Hq, Hkv, N, d = 1, 4, 2, 23, 6
    q, k, v = rnd(rng, B, Hq, N, d), rnd(rng, B, Hkv, N, d), rnd(rng, B, Hkv, N, d)
    dout = rnd(rng, B, Hq, N, d)
    lmk = p1_landmarks(k, Hq, Hq)
    s = oracle.Shape(B=B, Hq=Hq, Hkv=Hkv, Hl=Hq, N=N, L=N, d=d, chunk=1, topk=N, window=1, scale=0.4)
    r = oracle.fwd(s, q, k, v, lmk)
    g = oracle.bwd(s, dout, q, k, v, lmk, r["idx"])
    tq, tk, tv = _torch_dense_grads(q, k, v, dout, 0.4)
    np.testing.assert_allclose(g["dq"], tq, atol=1e-11)
    np.testing.assert_allclose(g["dv"], tv, atol=1e-11)
    dl = g["dlmk"].reshape(B, Hkv, Hq // Hkv, N, d).sum(2)
    np.testing.assert_allclose(g["dk"] + dl, tk, atol=1e-11)


def test_p7_backward_exact_mass_construction_matches_dense():
    """P7 under P2 (S=4, W=6): the gradient reaching each chunk's shared key
    kappa_c (token path summed over the chunk plus the landmark path) equals
    the dense-attention gradient of the tied keys."""
    rng = np.random.default_rng(27)
    B, Hq, Hkv, N, d, S, W = 1, 2, 1, 32, 5, 4, 6
    kappa, k, lmk, bias = p2_construction(rng, B, Hq, Hkv, Hq, N, d, S)
    q, v, dout = rnd(rng, B, Hq, N, d), rnd(rng, B, Hkv, N, d), rnd(rng, B, Hq, N, d)
    s = oracle.Shape(B=B, Hq=Hq, Hkv=Hkv, Hl=Hq, N=N, L=N, d=d, chunk=S, topk=N // S, window=W, scale=0.5)
    r = oracle.fwd(s, q, k, v, lmk, bias=bias)
    g = oracle.bwd(s, dout, q, k, v, lmk, r["idx"], bias=bias)
    tq, tk, tv = _torch_dense_grads(q, k, v, dout, 0.5)
    np.testing.assert_allclose(g["dq"], tq, atol=2e-6)
    np.testing.assert_allclose(g["dv"], tv, atol=2e-6)
    dkappa = g["dk"].reshape(B, Hkv, N // S, S, d).sum(3) + g["dlmk"].reshape(B, Hkv, Hq // Hkv, N // S, d).sum(2)
    tkappa = tk.reshape(B, Hkv, N // S, S, d).sum(3)
    np.testing.assert_allclose(dkappa, tkappa, atol=2e-6)


def test_backward_row_subset_is_additive():
    """The row-subset mode (used for sampled checks at full size) partitions the
    gradient: the sum over a split of the rows equals the all-rows result."""
    rng = np.random.default_rng(8)
    B, Hq, Hkv, N, d, S, W, K = 2, 4, 2, 40, 8, 4, 6, 3
    q, k, v = rnd(rng, B, Hq, N, d), rnd(rng, B, Hkv, N, d), rnd(rng, B, Hkv, N, d)
    lmk, dout = rnd(rng, B, Hq, N // S, d), rnd(rng, B, Hq, N, d)
    s = oracle.Shape(B=B, Hq=Hq, Hkv=Hkv, Hl=Hq, N=N, L=N, d=d, chunk=S, topk=K, window=W, scale=0.3)
    idx = oracle.fwd(s, q, k, v, lmk)["idx"]
    full = oracle.bwd(s, dout, q, k, v, lmk, idx)
    rows = np.array([(b, n) for b in range(B) for n in range(N)], np.int32)
    a = oracle.bwd(s, dout, q, k, v, lmk, idx, rows=rows[::2])
    bb = oracle.bwd(s, dout, q, k, v, lmk, idx, rows=rows[1::2])
    for key in ("dq", "dk", "dv", "dlmk", "dbias"):
        np.testing.assert_allclose(a[key] + bb[key], full[key], atol=1e-12)
