"""The five synthetic workloads of the operator, named by what they are.

Shapes mirror the paper's long-context settings (chunk S = 64, local window
W = 512, top-K 16/32, GQA groups of 4); inputs are i.i.d. N(0, 1).  Landmark
heads Hl = Hq (one compressed key per query head, Appendix C).  For decode
the caller has already appended the new token, so the query sits at position
``ctx`` and the valid length is ``ctx + 1``; the cache capacity L is that
length rounded up to whole chunks.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace


@dataclass(frozen=True)
class Workload:
    name: str
    wid: int          # seed namespace
    kind: str         # "prefill", "decode" or "train"
    B: int
    Hq: int
    Hkv: int
    d: int
    N: int            # queries per sequence (decode: 1)
    L: int            # key capacity per sequence
    chunk: int
    topk: int
    window: int
    dtype: str        # "f32" or "bf16"
    Hl: int = 0       # landmark heads; 0 means Hq
    ctx: int = 0      # decode: cached tokens before the new one

    @property
    def landmark_heads(self) -> int:
        return self.Hl or self.Hq

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    @property
    def nchunks(self) -> int:
        return self.L // self.chunk

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


def _decode(name, wid, B, ctx, topk):
    L = ((ctx + 1 + 63) // 64) * 64
    return Workload(name, wid, "decode", B=B, Hq=32, Hkv=8, d=128, N=1, L=L, chunk=64, topk=topk, window=512,
                    dtype="bf16", ctx=ctx)


WORKLOADS = {
    w.name: w
    for w in [
        Workload("prefill_2k_f32_tiny", 1, "prefill", B=1, Hq=4, Hkv=1, d=64, N=2048, L=2048, chunk=64, topk=4,
                 window=512, dtype="f32"),
        Workload("prefill_32k_bf16", 2, "prefill", B=1, Hq=32, Hkv=8, d=128, N=32768, L=32768, chunk=64, topk=16,
                 window=512, dtype="bf16"),
        _decode("decode_131k_bf16_b32", 3, B=32, ctx=131072, topk=16),
        _decode("decode_1m_bf16_b4", 4, B=4, ctx=1048576, topk=32),
        Workload("train_16k_bf16_b4", 5, "train", B=4, Hq=32, Hkv=8, d=128, N=16384, L=16384, chunk=64, topk=16,
                 window=512, dtype="bf16"),
    ]
}
