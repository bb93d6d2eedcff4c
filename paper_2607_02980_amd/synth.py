"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module holds no arithmetic of the attention method: it only draws seeded
N(0, 1) tensors (i.i.d., or correlated along the sequence for the locality
inputs) and rounds them to the storage dtype.
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


def ar1_host(shape, seed: int, dtype: str = "f32", rho: float = 0.97, device="cpu") -> torch.Tensor:
    """Seeded N(0, 1) marginals correlated along the second-to-last axis (the
    sequence axis of [B, H, N, d]): x_0 = e_0, x_i = rho x_{i-1} + sqrt(1 - rho^2) e_i
    with e i.i.d. N(0, 1).  Adjacent queries drawn this way retrieve overlapping
    chunks, as the queries of a trained model do (rho = 0.97 gives a chunk-overlap
    ratio of about 0.86 for 16 adjacent queries at top-16).  The noise is drawn on
    the host; the recursion runs on ``device`` (float64 on the host, float32 on a
    GPU).  Rounded to ``dtype`` and returned on ``device`` as float32."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    ft = torch.float64 if str(device) == "cpu" else torch.float32
    e = torch.randn(*shape, generator=g, dtype=torch.float64).to(device=device, dtype=ft)
    x = torch.empty_like(e)
    c = (1.0 - rho * rho) ** 0.5
    n = shape[-2]
    # the recursion over blocks of T steps: inside a block, x = A (c e) + rho^(i+1) x_prev
    # with A[i][j] = rho^(i-j) for j <= i
    T = 256
    i = torch.arange(T, dtype=ft, device=device)
    A = torch.tril(rho ** (i[:, None] - i[None, :]).clamp(min=0)) * (i[:, None] >= i[None, :])
    decay = (rho ** (i + 1))[:, None]
    prev = None
    for t0 in range(0, n, T):
        t1 = min(n, t0 + T)
        blk = torch.matmul(A[: t1 - t0, : t1 - t0], c * e[..., t0:t1, :])
        if prev is None:
            blk = blk + (e[..., :1, :] - c * e[..., :1, :]) * decay[: t1 - t0] / rho  # x_0 = e_0
        else:
            blk = blk + decay[: t1 - t0] * prev
        x[..., t0:t1, :] = blk
        prev = blk[..., -1:, :]
    return round_to(x.to(torch.float32), dtype)


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
