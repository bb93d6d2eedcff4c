"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module holds no arithmetic of the attention method: it only draws i.i.d.
N(0, 1) tensors from seeded generators and rounds them to the storage dtype.
Both the oracle and the GPU library receive exactly these values.

Seeds follow one rule: ``seed = 1000 * workload_id + 10 * tensor_id + slab``
with tensor ids q=1, k=2, v=3, lmk=4, bias=5, dout=6, q_route=7.
"""
from __future__ import annotations

import torch

TENSOR_IDS = {"q": 1, "k": 2, "v": 3, "lmk": 4, "bias": 5, "dout": 6, "q_route": 7, "page_table": 8}


def seed_for(workload_id: int, tensor: str, slab: int = 0) -> int:
    return 1000 * workload_id + 10 * TENSOR_IDS[tensor] + slab


def round_to(t: torch.Tensor, dtype: str) -> torch.Tensor:
    """Round a float32 tensor to the storage dtype (RNE for bf16) and widen it back."""
    if dtype == "bf16":
        return t.to(torch.bfloat16).to(torch.float32)
    if dtype == "f32":
        return t
    raise ValueError(dtype)


def normal_host(shape, seed: int, dtype: str = "f32", std: float = 1.0) -> torch.Tensor:
    """N(0, std^2) on the host from ``torch.Generator('cpu')``, rounded to ``dtype``;
    returned as a float32 CPU tensor holding exactly the stored values."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    t = torch.randn(*shape, generator=g, dtype=torch.float32)
    if std != 1.0:
        t = t * std
    return round_to(t, dtype)


def normal_device(shape, seed: int, dtype: str, device) -> torch.Tensor:
    """N(0, 1) drawn directly on ``device`` with torch's seeded device generator
    (used for the multi-GB decode caches, where host generation and the copy
    would dominate).  Returned in the storage dtype; read back any slice with
    ``.float().cpu()`` to obtain exactly the stored values."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    t = torch.empty(*shape, dtype=tdt, device=device)
    t.normal_(0.0, 1.0, generator=g)
    return t


def torch_dtype(dtype: str):
    return torch.bfloat16 if dtype == "bf16" else torch.float32
