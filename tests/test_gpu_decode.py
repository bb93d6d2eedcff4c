"""GPU parity of hils_decode_fwd against the oracle (query at seqlens[b]-1).

Covers unequal sequence lengths in one batch (including a single-token
sequence and a full cache), seqlens = NULL (full capacity), Q-Cal routing and
bias, Hl = Hkv, forced-index mode, and both bf16 decode layouts (a workgroup per
row from 256 rows up, per-part workgroups below)."""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_helpers import (check_close, check_lse, check_selection, host_inputs, log, np32, oshape, to_device)

pytestmark = pytest.mark.gpu

CASES = {
    "bf16_ragged_lengths": (dict(B=4, Hq=8, Hkv=2, N=1, L=4096, d=128, topk=8, window=512), 201, False, False,
                            [4096, 1, 2500, 577]),
    "bf16_full_capacity": (dict(B=2, Hq=32, Hkv=8, N=1, L=8192, d=128, topk=16, window=512), 202, False, False, None),
    "f32_route_bias_Hl_eq_Hkv": (dict(B=3, Hq=8, Hkv=1, Hl=1, N=1, L=3072, d=64, topk=32, window=100, dtype="f32"),
                                 203, True, True, [3072, 3000, 65]),
    "bf16_window1_G2": (dict(B=2, Hq=4, Hkv=2, N=1, L=2048, d=64, topk=5, window=1), 204, True, False, [2048, 2047]),
    # 256 (sequence, KV group) rows: the one-workgroup-per-row pass (fewer rows take
    # the per-part workgroups and a separate fusion pass)
    "bf16_many_rows_ragged": (dict(B=64, Hq=16, Hkv=4, N=1, L=1024, d=128, topk=8, window=256), 205, True, False,
                              [1024 - 13 * i for i in range(63)] + [1]),
    # the paper's efficiency shape (Sec. 7.1): d = 64, 16 query / 2 KV heads, K = 32, W = 512
    "bf16_paper_shape_d64_G8_K32": (dict(B=4, Hq=16, Hkv=2, N=1, L=8192, d=64, topk=32, window=512), 206, False,
                                    False, [8192, 5000, 2600, 700]),
    "bf16_K64": (dict(B=3, Hq=8, Hkv=2, N=1, L=8192, d=128, topk=64, window=256), 207, False, False,
                 [8192, 4500, 4097]),
    # one landmark head 150 above the rest of its group (per-head fusion weights)
    "bf16_head_gap_150": (dict(B=4, Hq=8, Hkv=2, N=1, L=4096, d=128, topk=8, window=512), 208, False, False,
                          [4096, 3000, 1500, 600]),
    "bf16_head_gap_150_many_rows": (dict(B=64, Hq=16, Hkv=4, N=1, L=1024, d=64, topk=8, window=128), 209, False,
                                    False, [1024 - 13 * i for i in range(64)]),
    # one landmark head per KV group with G <= 4 heads: the scan reads each landmark
    # row once and scores it against the group's heads (several slices, ragged)
    "bf16_route_bias_Hl_eq_Hkv_G4": (dict(B=3, Hq=8, Hkv=2, Hl=2, N=1, L=20480, d=128, topk=16, window=512), 210,
                                     True, True, [20480, 9000, 300]),
    "bf16_Hl_eq_Hkv_G2_d64": (dict(B=2, Hq=4, Hkv=2, Hl=2, N=1, L=8192, d=64, topk=8, window=256), 211, False, False,
                              [8192, 4100]),
    "f32_Hl_eq_Hkv_G4": (dict(B=2, Hq=4, Hkv=1, Hl=1, N=1, L=4096, d=64, topk=8, window=128, dtype="f32"), 212, True,
                         False, [4096, 1800]),
}
HEAD_GAP = {"bf16_head_gap_150": (1, 150.0), "bf16_head_gap_150_many_rows": (6, 150.0)}


def run_case(name, forced=False, flags=0):
    from paper_2607_02980_amd import hils

    kw, wid, bias, route, seqlens = CASES[name]
    p = hils.Params(flags=flags, **kw)
    log(f"[decode] case={name} forced={forced} seqlens={seqlens} params={kw}")
    host = host_inputs(p, wid, bias=bias, route=route, head_gap=HEAD_GAP.get(name))
    dev = to_device(host, p)
    qpos = np.array([[(sl if seqlens else p.L) - 1] for sl in (seqlens or [p.L] * p.B)], np.int32)
    sl_dev = torch.tensor(seqlens, dtype=torch.int32, device="cuda") if seqlens else None
    s = oshape(p)
    ref = oracle.fwd(s, np32(host["q"]), np32(host["k"]), np32(host["v"]), np32(host["lmk"]),
                     bias=np32(host.get("bias")), q_route=np32(host.get("q_route")), qpos=qpos)
    idx_in = None
    if forced:
        p.flags = hils.HILS_FLAG_GIVEN_IDX | flags
        idx_in = torch.from_numpy(ref["idx"]).cuda()
    out, lse, idx = hils.hils_decode_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"], dev.get("bias"),
                                         dev.get("q_route"), sl_dev, idx=idx_in)
    torch.cuda.synchronize()
    gidx = idx.cpu().numpy()
    ndiff = check_selection(p, host, gidx, ref["idx"], qpos=qpos)
    log(f"  selection: {ndiff} rows differ only by accepted ties")
    if ndiff:
        ref = oracle.fwd(s, np32(host["q"]), np32(host["k"]), np32(host["v"]), np32(host["lmk"]),
                         bias=np32(host.get("bias")), q_route=np32(host.get("q_route")), qpos=qpos, idx=gidx)
    check_close("out", np32(out), ref["out"], p.dtype)
    check_lse(np32(lse), ref["lse"], p.dtype)


@pytest.mark.parametrize("name", list(CASES))
def test_decode_matches_oracle(name):
    run_case(name)


def test_decode_forced_index():
    run_case("bf16_ragged_lengths", forced=True)


def test_decode_forced_index_many_rows():
    run_case("bf16_many_rows_ragged", forced=True)


@pytest.mark.parametrize("name", list(CASES))
def test_decode_head_normalised_selection(name):
    from paper_2607_02980_amd import hils

    run_case(name, flags=hils.HILS_FLAG_HEAD_NORM_SELECT)
