"""GPU parity of hils_bwd against the oracle's backward (selection fixed to the
forward's idx), every gradient element compared: dq, dk, dv, dk' (dlmk), db'
(dlmk_bias) and dq^ (dq_route)."""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_helpers import check_close, host_inputs, log, np32, oshape, to_device

pytestmark = pytest.mark.gpu

CASES = {
    "f32_small": (dict(B=1, Hq=4, Hkv=1, N=512, L=512, d=64, topk=4, window=128, dtype="f32"), 301, False, False),
    "bf16_ragged_route_bias": (dict(B=2, Hq=8, Hkv=2, N=640, L=640, d=128, topk=8, window=200), 302, True, True),
    "bf16_Hl_eq_Hkv_window1": (dict(B=1, Hq=8, Hkv=2, Hl=2, N=768, L=768, d=64, topk=6, window=1), 303, True, False),
    "f32_G8_bias_boosted": (dict(B=1, Hq=8, Hkv=1, N=600, L=640, d=128, topk=5, window=64, dtype="f32"), 304, True,
                            True),
    "bf16_G8_route_bias_ragged": (dict(B=1, Hq=8, Hkv=1, N=600, L=640, d=128, topk=5, window=64), 305, True, True),
    "bf16_G1_d64": (dict(B=2, Hq=2, Hkv=2, N=500, L=512, d=64, topk=3, window=70), 306, False, False),
    "bf16_G2_Hl_eq_Hkv_topk_exceeds": (dict(B=1, Hq=4, Hkv=2, Hl=2, N=1100, L=1152, d=128, topk=16, window=100),
                                       307, True, False),
    "bf16_G8_Hl_eq_Hkv_d64": (dict(B=1, Hq=8, Hkv=1, Hl=1, N=400, L=448, d=64, topk=4, window=64), 308, False,
                              False),
    "bf16_all_local": (dict(B=1, Hq=4, Hkv=1, N=200, L=256, d=64, topk=4, window=512), 309, False, False),
    # bf16 at K = 32 and K = 64 (the per-slot dq partials and the chunk lists grow with K)
    "bf16_K32": (dict(B=1, Hq=8, Hkv=2, N=2500, L=2560, d=128, topk=32, window=256), 310, False, False),
    "bf16_K64_d64_route_bias": (dict(B=1, Hq=4, Hkv=1, N=4500, L=4544, d=64, topk=64, window=64), 311, True, True),
    # the paper's efficiency shape (Sec. 7.1): d = 64, 16 query / 2 KV heads, K = 32, W = 512
    "bf16_paper_shape_d64_G8_K32": (dict(B=1, Hq=16, Hkv=2, N=4096, L=4096, d=64, topk=32, window=512), 312, False,
                                    False),
    # one landmark head 150 above the rest of its group (per-head fusion weights)
    "bf16_head_gap_150": (dict(B=1, Hq=8, Hkv=2, N=1100, L=1152, d=128, topk=8, window=128), 313, False, False),
}
HEAD_GAP = {"bf16_head_gap_150": (1, 150.0)}


def run_case(name):
    from paper_2607_02980_amd import hils

    kw, wid, bias, route = CASES[name]
    p = hils.Params(**kw)
    log(f"[bwd] case={name} params={kw}")
    host = host_inputs(p, wid, bias=bias, route=route, dout=True, bias_shift=2.0 if bias else 0.0,
                       head_gap=HEAD_GAP.get(name))
    dev = to_device(host, p)
    out, lse, idx = hils.hils_prefill_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"], dev.get("bias"),
                                          dev.get("q_route"))
    g = hils.hils_bwd(p, dev["dout"], dev["q"], dev["k"], dev["v"], dev["lmk"], out, lse, idx, dev.get("bias"),
                      dev.get("q_route"))
    torch.cuda.synchronize()
    s = oshape(p)
    ref = oracle.bwd(s, np32(host["dout"]), np32(host["q"]), np32(host["k"]), np32(host["v"]), np32(host["lmk"]),
                     idx.cpu().numpy(), bias=np32(host.get("bias")), q_route=np32(host.get("q_route")))
    for key, rkey in (("dq", "dq"), ("dk", "dk"), ("dv", "dv"), ("dlmk", "dlmk"), ("dlmk_bias", "dbias"),
                      ("dq_route", "dq_route")):
        if ref[rkey] is None:
            continue
        check_close(key, np32(g[key]), ref[rkey], p.dtype, rel=True)
    return g


@pytest.mark.parametrize("name", list(CASES))
def test_bwd_matches_oracle(name):
    run_case(name)


def test_bwd_is_deterministic():
    from paper_2607_02980_amd import hils

    kw, wid, bias, route = CASES["bf16_ragged_route_bias"]
    p = hils.Params(**kw)
    dev = to_device(host_inputs(p, wid, bias=True, route=True, dout=True), p)
    out, lse, idx = hils.hils_prefill_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"], dev["bias"], dev["q_route"])
    a = hils.hils_bwd(p, dev["dout"], dev["q"], dev["k"], dev["v"], dev["lmk"], out, lse, idx, dev["bias"],
                      dev["q_route"])
    b = hils.hils_bwd(p, dev["dout"], dev["q"], dev["k"], dev["v"], dev["lmk"], out, lse, idx, dev["bias"],
                      dev["q_route"])
    torch.cuda.synchronize()
    for key in a:
        assert torch.equal(a[key], b[key]), key
