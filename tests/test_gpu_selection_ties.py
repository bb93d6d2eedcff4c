"""Exact ties in the selection (Eq. (9) rank with ties to the smaller chunk).

Landmark rows are copies of a few class vectors (every chunk takes one class at
random, the same class for every head), so the group scores of a row tie
exactly inside a class, on the GPU (identical arithmetic per chunk) as in the
oracle.  The GPU selection must then equal the oracle's exactly, ids included:
among equal scores the smaller chunk ids win.  One class makes every candidate
tie; 3 classes tie large groups (more survivors than a wavefront holds); 40
classes tie a few entries per class."""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_helpers import host_inputs, log, np32, oshape, to_device

pytestmark = pytest.mark.gpu


def class_landmarks(p, host, n_classes, seed):
    rng = np.random.default_rng(seed)
    nc = p.L // p.chunk
    Hl = p.Hl or p.Hq
    vecs = np32(host["lmk"])[:, :, :n_classes].copy()  # [B, Hl, n_classes, d]: bf16-exact values
    cls = rng.integers(0, n_classes, size=(p.B, nc))
    lmk = np.empty((p.B, Hl, nc, p.d), np.float32)
    for b in range(p.B):
        lmk[b] = vecs[b][:, cls[b]]
    host = dict(host)
    host["lmk"] = torch.from_numpy(lmk)
    return host


@pytest.mark.parametrize("n_classes", [1, 3, 40])
def test_prefill_ties_go_to_smaller_chunks(n_classes):
    from paper_2607_02980_amd import hils

    p = hils.Params(B=1, Hq=8, Hkv=2, N=3072, L=3072, d=128, topk=16, window=256)
    host = class_landmarks(p, host_inputs(p, 501), n_classes, 501)
    log(f"[ties] prefill classes={n_classes}")
    dev = to_device(host, p)
    _, _, idx = hils.hils_prefill_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"])
    torch.cuda.synchronize()
    rows = np.array([(0, n) for n in range(0, p.N, 7)], np.int32)
    ref = oracle.fwd(oshape(p), np32(host["q"]), np32(host["k"]), np32(host["v"]), np32(host["lmk"]), rows=rows)
    g = idx.cpu().numpy()
    for _, n in rows:
        np.testing.assert_array_equal(g[0, :, n], ref["idx"][0, :, n], err_msg=f"row {n}")


@pytest.mark.parametrize("n_classes", [1, 3, 40])
def test_decode_ties_go_to_smaller_chunks(n_classes):
    from paper_2607_02980_amd import hils

    p = hils.Params(B=4, Hq=8, Hkv=2, N=1, L=65536, d=128, topk=16, window=512)
    host = class_landmarks(p, host_inputs(p, 502), n_classes, 502)
    log(f"[ties] decode classes={n_classes}")
    dev = to_device(host, p)
    seqlens = [65536, 40000, 20001, 3000]
    sl = torch.tensor(seqlens, dtype=torch.int32, device="cuda")
    _, _, idx = hils.hils_decode_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"], seqlens=sl)
    torch.cuda.synchronize()
    ref = oracle.decode(oshape(p), np32(host["q"]), np32(host["k"]), np32(host["v"]), np32(host["lmk"]),
                        seqlens=seqlens)
    np.testing.assert_array_equal(idx.cpu().numpy(), ref["idx"])
