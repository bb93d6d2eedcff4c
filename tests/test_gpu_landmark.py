"""GPU parity of hils_landmark_fwd / hils_landmark_bwd (Prop. 3.1's landmark
compression and its backward) against the oracle, every element compared,
including the full 32K prefill shape (all 512 chunks of all 32 landmark heads)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_02980_amd import synth
from paper_2607_02980_amd.configs import WORKLOADS
from tests.gpu_helpers import check_close, log, np32, oshape

pytestmark = pytest.mark.gpu

CASES = {
    # name: (params, seed namespace)
    "bf16_d128_G4_per_head": (dict(B=2, Hq=8, Hkv=2, N=1, L=512, d=128), 401),
    "bf16_d64_Hl_eq_Hkv": (dict(B=1, Hq=8, Hkv=2, Hl=2, N=1, L=384, d=64), 402),
    "bf16_d64_G8": (dict(B=1, Hq=8, Hkv=1, N=1, L=256, d=64), 403),
    "f32_d64_G2": (dict(B=1, Hq=4, Hkv=2, N=1, L=256, d=64, dtype="f32"), 404),
    "f32_d128_G1": (dict(B=1, Hq=2, Hkv=2, N=1, L=192, d=128, dtype="f32"), 405),
}


def shared(p):
    from paper_2607_02980_amd import hils

    return bool(p.flags & hils.HILS_FLAG_SHARED_LMK_QUERY)


def inputs(p, wid, sd_q=2.0):
    nc = p.L // p.chunk
    Hl = p.Hl or p.Hq
    lq_shape = (Hl, p.d) if shared(p) else (p.B, Hl, nc, p.d)
    lq = synth.normal_device(lq_shape, synth.seed_for(wid, "q"), p.dtype, "cuda")
    lq = (lq.float() * sd_q).to(lq.dtype)  # sharper chunk attention than N(0,1)
    k = synth.normal_device((p.B, p.Hkv, p.L, p.d), synth.seed_for(wid, "k"), p.dtype, "cuda")
    dl = synth.normal_device((p.B, Hl, nc, p.d), synth.seed_for(wid, "dout"), p.dtype, "cuda")
    db = synth.normal_device((p.B, Hl, nc), synth.seed_for(wid, "bias"), "f32", "cuda")
    return lq, k, dl, db


def run(p, wid):
    from paper_2607_02980_amd import hils

    lq, k, dl, db = inputs(p, wid)
    lmk, bias = hils.hils_landmark_fwd(p, lq, k)
    dlq, dk = hils.hils_landmark_bwd(p, lq, k, dl, db)
    torch.cuda.synchronize()
    s = oshape(p)
    sh = shared(p)
    ref = oracle.landmark_fwd(s, np32(lq), np32(k), shared=sh)
    check_close("lmk", np32(lmk), ref["lmk"], p.dtype)
    # b' is float32 output; inputs are exact on both sides, the sums differ in order only
    d = np.abs(np32(bias) - ref["bias"]).max()
    log(f"  bias: max|d|={d:.3e}")
    assert d < (2e-4 if p.dtype == "bf16" else 1e-4), d
    g = oracle.landmark_bwd(s, np32(lq), np32(k), np32(dl), np32(db), shared=sh)
    check_close("dlq", np32(dlq), g["dlq"], p.dtype, rel=True)
    check_close("dk", np32(dk), g["dk"], p.dtype, rel=True)


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("query", ["per_chunk", "shared"])
def test_landmark_matches_oracle(name, query):
    from paper_2607_02980_amd import hils

    kw, wid = CASES[name]
    flags = hils.HILS_FLAG_SHARED_LMK_QUERY if query == "shared" else 0
    p = hils.Params(topk=1, window=1, flags=flags, **kw)
    log(f"[landmark] case={name} query={query} params={kw}")
    run(p, wid)


@pytest.mark.parametrize("query", ["per_chunk", "shared"])
def test_landmark_full_prefill_shape(query):
    from paper_2607_02980_amd import hils

    W = WORKLOADS["prefill_32k_bf16"]
    flags = hils.HILS_FLAG_SHARED_LMK_QUERY if query == "shared" else 0
    p = hils.Params(B=W.B, Hq=W.Hq, Hkv=W.Hkv, N=1, L=W.L, d=W.d, chunk=W.chunk, topk=1, window=1, dtype=W.dtype,
                    flags=flags)
    log(f"[landmark] full shape of {W.name}: B={p.B} Hl={p.Hl or p.Hq} chunks={p.L // p.chunk} d={p.d}")
    run(p, 406)


def test_landmark_is_deterministic():
    from paper_2607_02980_amd import hils

    kw, wid = CASES["bf16_d128_G4_per_head"]
    p = hils.Params(topk=1, window=1, **kw)
    lq, k, dl, db = inputs(p, wid)
    a = hils.hils_landmark_fwd(p, lq, k) + hils.hils_landmark_bwd(p, lq, k, dl, db)
    b = hils.hils_landmark_fwd(p, lq, k) + hils.hils_landmark_bwd(p, lq, k, dl, db)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)
