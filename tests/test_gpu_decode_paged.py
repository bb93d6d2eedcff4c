"""GPU parity of the decode step with N > 1 new queries per sequence (drafted
tokens verified together) and of hils_decode_paged_fwd (one chunk per page,
pages permuted in the pool, unused pages, a prefix shared by two sequences)
against the oracle.

Inputs: the seeded N(0,1) caches of host_inputs, cut into pages on the host.
The oracle gets the pools and the page table (it gathers them back itself);
the tie-aware selection check reads the equivalent contiguous caches."""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_helpers import (check_close, check_lse, check_selection, host_inputs, log, np32, oshape, to_device)

pytestmark = pytest.mark.gpu

# name: (params, workload id, bias, route, seqlens, paged)
CASES = {
    "bf16_multi_token_ragged": (dict(B=3, Hq=8, Hkv=2, N=4, L=4096, d=128, topk=8, window=512), 301, False, False,
                                [4096, 2, 1700], False),
    "bf16_paged_single_token": (dict(B=3, Hq=32, Hkv=8, N=1, L=4096, d=128, topk=16, window=512), 302, False, False,
                                [4096, 3000, 577], True),
    "bf16_paged_multi_token_G8": (dict(B=2, Hq=8, Hkv=1, N=3, L=3072, d=64, topk=16, window=300), 303, True, False,
                                  [3072, 1500], True),
    "f32_paged_route_bias_Hl_eq_Hkv": (dict(B=3, Hq=8, Hkv=2, Hl=2, N=2, L=2048, d=64, topk=5, window=100,
                                            dtype="f32"), 304, True, True, [2048, 1999, 130], True),
    "bf16_paged_window1_G1": (dict(B=2, Hq=4, Hkv=4, N=5, L=2048, d=64, topk=7, window=1), 305, False, True,
                              None, True),
    # one landmark head 150 above the rest of its group (per-head fusion weights),
    # several new queries per sequence sharing a workgroup, and a paged cache
    "bf16_multi_token_head_gap_150": (dict(B=2, Hq=8, Hkv=2, N=3, L=4096, d=128, topk=8, window=512), 307, False,
                                      False, [4096, 2100], False),
    "bf16_paged_multi_token_K32_d64_G8": (dict(B=2, Hq=16, Hkv=2, N=2, L=4096, d=64, topk=32, window=512), 308,
                                          False, False, [4096, 3500], True),
    # one landmark page row per KV group (Hl = Hkv, G = 4): read once for the group's heads
    "bf16_paged_Hl_eq_Hkv_G4": (dict(B=2, Hq=8, Hkv=2, Hl=2, N=1, L=16384, d=128, topk=16, window=512), 309, True,
                                True, [16384, 7000], True),
}
HEAD_GAP = {"bf16_multi_token_head_gap_150": (2, 150.0)}


def make_pool(p, host, rng):
    """Pools [P, ...] holding every chunk of every sequence at a random page, with 9
    unused pages; sequence B-1 shares its first chunks with sequence 0 when B > 1."""
    nc = p.L // p.chunk
    Hl = p.Hl or p.Hq
    shared = min(6, nc) if p.B > 1 else 0
    P = p.B * nc + 9
    perm = rng.permutation(P)
    table = perm[np.arange(p.B * nc).reshape(p.B, nc)].astype(np.int32)
    k, v, lmk = np32(host["k"]).copy(), np32(host["v"]).copy(), np32(host["lmk"]).copy()
    bias = np32(host["bias"]).copy() if "bias" in host else None
    if shared:
        S = p.chunk
        k[-1, :, :shared * S], v[-1, :, :shared * S] = k[0, :, :shared * S], v[0, :, :shared * S]
        lmk[-1, :, :shared] = lmk[0, :, :shared]
        if bias is not None:
            bias[-1, :, :shared] = bias[0, :, :shared]
        table[-1, :shared] = table[0, :shared]
    pools = {
        "k": rng.standard_normal((P, p.Hkv, p.chunk, p.d)).astype(np.float32),
        "v": rng.standard_normal((P, p.Hkv, p.chunk, p.d)).astype(np.float32),
        "lmk": rng.standard_normal((P, Hl, p.d)).astype(np.float32),
        "bias": rng.standard_normal((P, Hl)).astype(np.float32) if bias is not None else None,
    }
    for b in range(p.B):
        for c in range(nc):
            pg = table[b, c]
            pools["k"][pg] = k[b, :, c * p.chunk:(c + 1) * p.chunk]
            pools["v"][pg] = v[b, :, c * p.chunk:(c + 1) * p.chunk]
            pools["lmk"][pg] = lmk[b, :, c]
            if bias is not None:
                pools["bias"][pg] = bias[b, :, c]
    contiguous = dict(host, k=torch.from_numpy(k), v=torch.from_numpy(v), lmk=torch.from_numpy(lmk))
    if bias is not None:
        contiguous["bias"] = torch.from_numpy(bias)
    return pools, table, contiguous


def run_case(name, flags=0):
    from paper_2607_02980_amd import hils

    kw, wid, bias, route, seqlens, paged = CASES[name]
    p = hils.Params(flags=flags, **kw)
    log(f"[decode-paged] case={name} seqlens={seqlens} params={kw}")
    host = host_inputs(p, wid, bias=bias, route=route, head_gap=HEAD_GAP.get(name))
    s = oshape(p)
    sl_dev = torch.tensor(seqlens, dtype=torch.int32, device="cuda") if seqlens else None
    qpos = oracle.decode_positions(s, seqlens)
    route_h = np32(host.get("q_route"))
    if paged:
        pools, table, host = make_pool(p, host, np.random.default_rng(wid))
        ref = oracle.decode(s, np32(host["q"]), pools["k"], pools["v"], pools["lmk"], seqlens=seqlens,
                            bias=pools["bias"], q_route=route_h, block_table=table)
        dt = p.torch_dtype
        dp = {k_: (torch.from_numpy(x).to("cuda", torch.float32 if k_ == "bias" else dt) if x is not None else None)
              for k_, x in pools.items()}
        q = host["q"].to("cuda", dt)
        qr = host["q_route"].to("cuda", dt) if route else None
        out, lse, idx = hils.hils_decode_paged_fwd(p, q, dp["k"], dp["v"], dp["lmk"],
                                                   torch.from_numpy(table).cuda(), dp["bias"], qr, sl_dev)
    else:
        ref = oracle.decode(s, np32(host["q"]), np32(host["k"]), np32(host["v"]), np32(host["lmk"]), seqlens=seqlens,
                            bias=np32(host.get("bias")), q_route=route_h)
        dev = to_device(host, p)
        out, lse, idx = hils.hils_decode_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"], dev.get("bias"),
                                             dev.get("q_route"), sl_dev)
    torch.cuda.synchronize()
    gidx = idx.cpu().numpy()
    ndiff = check_selection(p, host, gidx, ref["idx"], qpos=qpos)
    log(f"  selection: {ndiff} rows differ only by accepted ties")
    if ndiff:
        ref = oracle.decode(s, np32(host["q"]), np32(host["k"]), np32(host["v"]), np32(host["lmk"]),
                            seqlens=seqlens, bias=np32(host.get("bias")), q_route=route_h, idx=gidx)
    check_close("out", np32(out), ref["out"], p.dtype)
    check_lse(np32(lse), ref["lse"], p.dtype)


@pytest.mark.parametrize("name", list(CASES))
def test_decode_paged_and_multi_token(name):
    run_case(name)


@pytest.mark.parametrize("name", ["bf16_multi_token_ragged", "bf16_paged_window1_G1"])
def test_decode_multi_token_head_normalised(name):
    # the two-pass scan with several new queries per sequence sharing its workgroups
    from paper_2607_02980_amd import hils

    run_case(name, flags=hils.HILS_FLAG_HEAD_NORM_SELECT)


def test_paged_equals_contiguous_bitwise():
    # the same caches, contiguous and paged: the kernels read the same values in
    # the same order, so the outputs agree bit for bit
    from paper_2607_02980_amd import hils

    p = hils.Params(B=2, Hq=8, Hkv=2, N=2, L=2048, d=128, topk=8, window=256)
    host = host_inputs(p, 306)
    pools, table, host = make_pool(p, host, np.random.default_rng(306))
    dev = to_device(host, p)
    sl = torch.tensor([2048, 1200], dtype=torch.int32, device="cuda")
    a = hils.hils_decode_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"], seqlens=sl)
    dp = {k_: torch.from_numpy(x).to("cuda", p.torch_dtype) for k_, x in pools.items() if x is not None}
    b = hils.hils_decode_paged_fwd(p, dev["q"], dp["k"], dp["v"], dp["lmk"], torch.from_numpy(table).cuda(),
                                   seqlens=sl)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)
