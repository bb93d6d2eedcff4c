"""Independent references used to pin the oracle: textbook dense causal
attention, naive block-sparse attention (Sec. 2.1, Eqs. (1)-(3)), brute-force
subset search, and the constructions under which HiLS reduces to them."""
from __future__ import annotations

import itertools
import math

import numpy as np


def dense_causal(q, k, v, scale, qpos=None):
    """Textbook causal softmax attention.  q [B,Hq,N,d], k/v [B,Hkv,L,d].
    Query n attends keys j <= pos(n).  Returns (out, lse)."""
    B, Hq, N, d = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    out = np.zeros(q.shape, np.float64)
    lse = np.zeros((B, Hq, N), np.float64)
    for b in range(B):
        for h in range(Hq):
            g = h // G
            s = scale * (q[b, h].astype(np.float64) @ k[b, g].astype(np.float64).T)
            for n in range(N):
                i = n if qpos is None else int(qpos[b, n])
                row = s[n, : i + 1]
                m = row.max()
                e = np.exp(row - m)
                out[b, h, n] = (e / e.sum()) @ v[b, g, : i + 1].astype(np.float64)
                lse[b, h, n] = m + math.log(e.sum())
    return out, lse


def naive_bsa(q, k, v, scale, chunk, window, topk):
    """Naive block-sparse attention (Sec. 2.1): exact chunk masses Z_c (Eq. (1)),
    top-K by Z_c (Eq. (2)), weights exp(s_ij) / calZ over selected tokens and the
    window (Eq. (3)).  MHA only (one selection per head).  Returns (out, idx)."""
    B, H, N, d = q.shape
    out = np.zeros(q.shape, np.float64)
    idx = np.full((B, H, N, topk), -1, np.int64)
    for b in range(B):
        for h in range(H):
            s = scale * (q[b, h].astype(np.float64) @ k[b, h].astype(np.float64).T)
            for i in range(N):
                ell = max(0, (i - window + 1) // chunk) * chunk
                ncand = ell // chunk
                Z = np.array([np.exp(s[i, c * chunk:(c + 1) * chunk]).sum() for c in range(ncand)])
                order = sorted(range(ncand), key=lambda c: (-Z[c], c))[:topk]
                sel = sorted(order)
                idx[b, h, i, : len(sel)] = sel
                keys = list(range(ell, i + 1))
                for c in sel:
                    keys += list(range(c * chunk, (c + 1) * chunk))
                keys = np.array(sorted(keys))
                w = np.exp(s[i, keys])
                w /= w.sum()
                out[b, h, i] = w @ v[b, h, keys].astype(np.float64)
    return out, idx


def brute_force_topk(sigma, K):
    """All subsets of size min(K, n); returns the list of maximisers of sum(sigma)."""
    n = len(sigma)
    m = min(K, n)
    best, arg = -np.inf, []
    for sub in itertools.combinations(range(n), m):
        t = float(np.sum(sigma[list(sub)]))
        if t > best + 1e-12:
            best, arg = t, [sub]
        elif abs(t - best) <= 1e-12:
            arg.append(sub)
    return arg


def group_scores_np(q_route, lmk, bias, scale, b, g, i, n, G, Hl, Hq, ncand):
    """sigma_c = max over the group's heads of scale * q^ . k'_c + b'_c (Eq. (9), App. C)."""
    sig = np.full(ncand, -np.inf)
    for hh in range(G):
        h = g * G + hh
        hl = h if Hl == Hq else g
        s = scale * (lmk[b, hl, :ncand].astype(np.float64) @ q_route[b, h, n].astype(np.float64))
        if bias is not None:
            s = s + bias[b, hl, :ncand]
        sig = np.maximum(sig, s)
    return sig


def p1_landmarks(k, Hq, Hl):
    """P1: chunk size 1 and k'_c = k_c (for every landmark head of the group)."""
    B, Hkv, L, d = k.shape
    G = Hq // Hkv
    if Hl == Hkv:
        return k.copy()
    return np.repeat(k, G, axis=1).copy()


def p2_construction(rng, B, Hq, Hkv, Hl, L, d, S):
    """P2: keys constant inside each chunk (k_j = kappa_c), landmarks k'_c = kappa_c,
    bias b'_c = log S.  Then s^_c = log Z_c exactly."""
    G = Hq // Hkv
    nc = L // S
    kappa = rng.standard_normal((B, Hkv, nc, d)).astype(np.float32)
    k = np.repeat(kappa, S, axis=2).copy()
    lmk = kappa.copy() if Hl == Hkv else np.repeat(kappa, G, axis=1).copy()
    bias = np.full((B, Hl, nc), math.log(S), np.float32)
    return kappa, k, lmk, bias
