"""hils_decode_fwd_noalloc (the decode forward whose workspace is the library's
fixed per-GPU array) against hils_decode_fwd (the same kernels with a caller
workspace), through the C-ABI: two calls in a row, the second smaller than the
first, each compared with the workspace entry point (identical bits) and with
the oracle on sampled sequences (the parity tolerances)."""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_helpers import check_close, check_lse, check_selection, host_inputs, log, np32, oshape, to_device

pytestmark = pytest.mark.gpu

# (params, workload id, seqlens): the second call has fewer sequences, a shorter
# cache and fewer candidates, so it reads only part of what the first one wrote
CALLS = [
    (dict(B=8, Hq=32, Hkv=8, N=1, L=16384, d=128, topk=16, window=512), 401,
     [16384, 16000, 9000, 5000, 2049, 700, 64, 1]),
    (dict(B=3, Hq=8, Hkv=2, N=2, L=4096, d=64, topk=8, window=256), 402, [4096, 1500, 2]),
]


def test_noalloc_decode_matches_workspace_decode():
    from paper_2607_02980_amd import hils

    for kw, wid, seqlens in CALLS:
        p = hils.Params(**kw)
        need = hils.hils_workspace_size(p, hils.HILS_OP_DECODE)
        log(f"[noalloc] params={kw} seqlens={seqlens} workspace={need} bytes "
            f"(array {hils.HILS_DECODE_NOALLOC_SCRATCH_BYTES})")
        assert need <= hils.HILS_DECODE_NOALLOC_SCRATCH_BYTES
        host = host_inputs(p, wid, bias=True, route=True)
        dev = to_device(host, p)
        sl = torch.tensor(seqlens, dtype=torch.int32, device="cuda")
        a = hils.hils_decode_fwd_noalloc(p, dev["q"], dev["k"], dev["v"], dev["lmk"], dev["bias"], dev["q_route"], sl)
        b = hils.hils_decode_fwd(p, dev["q"], dev["k"], dev["v"], dev["lmk"], dev["bias"], dev["q_route"], sl)
        torch.cuda.synchronize()
        for name, x, y in zip(("out", "lse", "idx"), a, b):
            assert torch.equal(x, y), f"{name}: the no-allocation decode differs from hils_decode_fwd"
        # and the oracle, on three of the sequences
        s = oshape(p)
        pick = [0, len(seqlens) // 2, len(seqlens) - 1]
        ref = oracle.decode(s, np32(host["q"]), np32(host["k"]), np32(host["v"]), np32(host["lmk"]),
                            seqlens=seqlens, bias=np32(host["bias"]), q_route=np32(host["q_route"]))
        qpos = oracle.decode_positions(s, seqlens)
        gidx = a[2].cpu().numpy()
        rows = [(bb, n) for bb in pick for n in range(p.N)]
        ndiff = check_selection(p, host, gidx, ref["idx"], qpos=qpos, rows=rows)
        if ndiff:
            ref = oracle.decode(s, np32(host["q"]), np32(host["k"]), np32(host["v"]), np32(host["lmk"]),
                                seqlens=seqlens, bias=np32(host["bias"]), q_route=np32(host["q_route"]), idx=gidx)
        check_close("out", np32(a[0])[pick], ref["out"][pick], p.dtype)
        check_lse(np32(a[1])[pick], ref["lse"][pick], p.dtype)
