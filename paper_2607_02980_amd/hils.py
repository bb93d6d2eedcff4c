"""ctypes binding of libhils.so -- argument marshalling only.

The entry points keep the C names (``hils_prefill_fwd``, ``hils_decode_fwd``,
``hils_decode_fwd_noalloc``, ``hils_decode_paged_fwd``, ``hils_bwd``,
``hils_landmark_fwd``, ``hils_landmark_bwd``,
``hils_workspace_size``, ``hils_prefill_record_cap``, ``hils_last_error``, ``hils_version``).
They take torch tensors already resident on the GPU, check dtype, shape,
device and contiguity, allocate missing outputs and the workspace with
``torch.empty`` and pass raw pointers plus the current HIP stream.  Every step
of the computation runs in the library's HIP kernels; there is no fallback:
if ``libhils.so`` is missing or fails to load, importing this module raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

# HILS_LIB names another build of the same sources (the sanitizer build of the
# host code, libhils_san.so); by default the in-tree libhils.so
_LIB_PATH = os.environ.get("HILS_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhils.so")

HILS_F32, HILS_BF16 = 0, 1
HILS_OK, HILS_ERR_INVALID, HILS_ERR_UNSUPPORTED, HILS_ERR_WORKSPACE, HILS_ERR_HIP = range(5)
HILS_FLAG_GIVEN_IDX = 1
HILS_FLAG_SHARED_LMK_QUERY = 2
HILS_FLAG_HEAD_NORM_SELECT = 4
HILS_FLAG_UNION_PACKING = 8
HILS_OP_PREFILL, HILS_OP_DECODE, HILS_OP_BWD, HILS_OP_LANDMARK = 0, 1, 2, 3


class HilsError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"hils error {code}: {msg}")
        self.code = code


class hils_params(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int), ("Hq", ctypes.c_int), ("Hkv", ctypes.c_int), ("Hl", ctypes.c_int),
                ("N", ctypes.c_int), ("L", ctypes.c_int), ("d", ctypes.c_int), ("chunk", ctypes.c_int),
                ("topk", ctypes.c_int), ("window", ctypes.c_int), ("scale", ctypes.c_float),
                ("dtype", ctypes.c_int), ("flags", ctypes.c_uint)]


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is not built; run `python -m paper_2607_02980_amd.build`")
    lib = ctypes.CDLL(_LIB_PATH)
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    P = ctypes.POINTER(hils_params)
    lib.hils_version.restype = ctypes.c_int
    lib.hils_last_error.restype = ctypes.c_char_p
    lib.hils_workspace_size.argtypes = [P, ctypes.c_int, ctypes.POINTER(sz)]
    lib.hils_prefill_fwd.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.hils_decode_fwd.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.hils_decode_paged_fwd.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, ctypes.c_int, vp, vp, vp, vp, vp, sz, vp]
    lib.hils_decode_fwd_noalloc.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.hils_bwd.argtypes = [P] + [vp] * 17 + [sz, vp]
    lib.hils_landmark_fwd.argtypes = [P, vp, vp, vp, vp, vp]
    lib.hils_landmark_bwd.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.hils_prefill_record_cap.argtypes = [sz]
    lib.hils_prefill_record_cap.restype = sz
    lib.hils_timing_enable.argtypes = [ctypes.c_int]
    lib.hils_timing_read.argtypes = [ctypes.c_char_p, sz, ctypes.POINTER(ctypes.c_float),
                                     ctypes.POINTER(ctypes.c_int), ctypes.c_int, ctypes.POINTER(ctypes.c_int)]
    for f in (lib.hils_workspace_size, lib.hils_prefill_fwd, lib.hils_decode_fwd, lib.hils_decode_fwd_noalloc,
              lib.hils_bwd,
              lib.hils_landmark_fwd, lib.hils_landmark_bwd, lib.hils_timing_enable, lib.hils_timing_read):
        f.restype = ctypes.c_int
    return lib


LIB = _load()


@dataclass
class Params:
    """Python mirror of ``hils_params``."""
    B: int
    Hq: int
    Hkv: int
    N: int
    L: int
    d: int
    chunk: int = 64
    topk: int = 16
    window: int = 512
    scale: float | None = None
    dtype: str = "bf16"
    Hl: int = 0
    flags: int = 0

    def c(self) -> hils_params:
        return hils_params(self.B, self.Hq, self.Hkv, self.Hl or self.Hq, self.N, self.L, self.d, self.chunk,
                           self.topk, self.window, float(self.scale if self.scale is not None else self.d ** -0.5),
                           HILS_BF16 if self.dtype == "bf16" else HILS_F32, self.flags)

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32


def hils_version() -> int:
    return LIB.hils_version()


def hils_prefill_record_cap(nbytes: int = 0) -> int:
    """Set (nbytes > 0) and/or read the chunk-major prefill's cap on the per-slot
    records of one segment of rows; returns the previous cap."""
    return int(LIB.hils_prefill_record_cap(int(nbytes)))


def hils_last_error() -> str:
    return LIB.hils_last_error().decode()


def _check(rc: int):
    if rc != HILS_OK:
        raise HilsError(rc, hils_last_error())


def hils_workspace_size(p: Params, op: int) -> int:
    n = ctypes.c_size_t(0)
    cp = p.c()
    _check(LIB.hils_workspace_size(ctypes.byref(cp), op, ctypes.byref(n)))
    return n.value


def _ptr(t, name, shape=None, dtype=None, required=True):
    if t is None:
        if required:
            raise ValueError(f"{name} is required")
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    return ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _workspace(p: Params, op: int, workspace):
    n = hils_workspace_size(p, op)
    if workspace is None:
        workspace = torch.empty(max(n, 1), dtype=torch.uint8, device="cuda")
    if workspace.numel() < n:
        raise ValueError(f"workspace has {workspace.numel()} bytes, {n} needed")
    return workspace, n


def _shapes(p: Params):
    nc = p.L // p.chunk
    Hl = p.Hl or p.Hq
    return {"q": (p.B, p.Hq, p.N, p.d), "kv": (p.B, p.Hkv, p.L, p.d), "lmk": (p.B, Hl, nc, p.d),
            "bias": (p.B, Hl, nc), "lse": (p.B, p.Hq, p.N), "idx": (p.B, p.Hkv, p.N, p.topk)}


def hils_prefill_fwd(p: Params, q, k, v, lmk, lmk_bias=None, q_route=None, out=None, lse=None, idx=None,
                     workspace=None):
    """Prefill forward.  Returns (out, lse, idx).  With ``p.flags & HILS_FLAG_GIVEN_IDX``
    the given ``idx`` is consumed instead of selected."""
    S, dt = _shapes(p), p.torch_dtype
    if out is None:
        out = torch.empty(S["q"], dtype=dt, device=q.device)
    if lse is None:
        lse = torch.empty(S["lse"], dtype=torch.float32, device=q.device)
    if idx is None:
        if p.flags & HILS_FLAG_GIVEN_IDX:
            raise ValueError("HILS_FLAG_GIVEN_IDX needs idx")
        idx = torch.empty(S["idx"], dtype=torch.int32, device=q.device)
    ws, n = _workspace(p, HILS_OP_PREFILL, workspace)
    cp = p.c()
    _check(LIB.hils_prefill_fwd(
        ctypes.byref(cp), _ptr(q, "q", S["q"], dt), _ptr(k, "k", S["kv"], dt), _ptr(v, "v", S["kv"], dt),
        _ptr(lmk, "lmk", S["lmk"], dt), _ptr(lmk_bias, "lmk_bias", S["bias"], torch.float32, False),
        _ptr(q_route, "q_route", S["q"], dt, False), _ptr(out, "out", S["q"], dt),
        _ptr(lse, "lse", S["lse"], torch.float32), _ptr(idx, "idx", S["idx"], torch.int32),
        _ptr(ws, "workspace"), n, _stream()))
    return out, lse, idx


def hils_decode_fwd(p: Params, q, k_cache, v_cache, lmk_cache, lmk_bias=None, q_route=None, seqlens=None,
                    out=None, lse=None, idx=None, workspace=None):
    """Decode forward, N >= 1 new queries per sequence (query n at seqlens[b] - N + n).
    Returns (out, lse, idx)."""
    S, dt = _shapes(p), p.torch_dtype
    if out is None:
        out = torch.empty(S["q"], dtype=dt, device=q.device)
    if lse is None:
        lse = torch.empty(S["lse"], dtype=torch.float32, device=q.device)
    if idx is None:
        if p.flags & HILS_FLAG_GIVEN_IDX:
            raise ValueError("HILS_FLAG_GIVEN_IDX needs idx")
        idx = torch.empty(S["idx"], dtype=torch.int32, device=q.device)
    ws, n = _workspace(p, HILS_OP_DECODE, workspace)
    cp = p.c()
    _check(LIB.hils_decode_fwd(
        ctypes.byref(cp), _ptr(q, "q", S["q"], dt), _ptr(k_cache, "k_cache", S["kv"], dt),
        _ptr(v_cache, "v_cache", S["kv"], dt), _ptr(lmk_cache, "lmk_cache", S["lmk"], dt),
        _ptr(lmk_bias, "lmk_bias", S["bias"], torch.float32, False), _ptr(q_route, "q_route", S["q"], dt, False),
        _ptr(seqlens, "seqlens", (p.B,), torch.int32, False), _ptr(out, "out", S["q"], dt),
        _ptr(lse, "lse", S["lse"], torch.float32), _ptr(idx, "idx", S["idx"], torch.int32),
        _ptr(ws, "workspace"), n, _stream()))
    return out, lse, idx


HILS_DECODE_NOALLOC_SCRATCH_BYTES = 64 << 20


def hils_decode_fwd_noalloc(p: Params, q, k_cache, v_cache, lmk_cache, lmk_bias=None, q_route=None, seqlens=None,
                            out=None, lse=None, idx=None):
    """hils_decode_fwd without a workspace: the library's fixed per-GPU array
    (HILS_DECODE_NOALLOC_SCRATCH_BYTES) serves as the workspace.  Outputs not
    given are allocated here with torch.empty (the C call itself allocates
    nothing).  Returns (out, lse, idx)."""
    S, dt = _shapes(p), p.torch_dtype
    if out is None:
        out = torch.empty(S["q"], dtype=dt, device=q.device)
    if lse is None:
        lse = torch.empty(S["lse"], dtype=torch.float32, device=q.device)
    if idx is None:
        if p.flags & HILS_FLAG_GIVEN_IDX:
            raise ValueError("HILS_FLAG_GIVEN_IDX needs idx")
        idx = torch.empty(S["idx"], dtype=torch.int32, device=q.device)
    cp = p.c()
    _check(LIB.hils_decode_fwd_noalloc(
        ctypes.byref(cp), _ptr(q, "q", S["q"], dt), _ptr(k_cache, "k_cache", S["kv"], dt),
        _ptr(v_cache, "v_cache", S["kv"], dt), _ptr(lmk_cache, "lmk_cache", S["lmk"], dt),
        _ptr(lmk_bias, "lmk_bias", S["bias"], torch.float32, False), _ptr(q_route, "q_route", S["q"], dt, False),
        _ptr(seqlens, "seqlens", (p.B,), torch.int32, False), _ptr(out, "out", S["q"], dt),
        _ptr(lse, "lse", S["lse"], torch.float32), _ptr(idx, "idx", S["idx"], torch.int32), _stream()))
    return out, lse, idx


def hils_decode_paged_fwd(p: Params, q, k_pages, v_pages, lmk_pages, block_table, bias_pages=None, q_route=None,
                          seqlens=None, out=None, lse=None, idx=None, workspace=None):
    """Decode forward over paged pools (one chunk per page): k/v_pages [P, Hkv, S, d],
    lmk_pages [P, Hl, d], bias_pages [P, Hl] f32, block_table [B, L/S] int32.
    Returns (out, lse, idx)."""
    S, dt = _shapes(p), p.torch_dtype
    P = k_pages.shape[0]
    Hl = p.Hl or p.Hq
    if out is None:
        out = torch.empty(S["q"], dtype=dt, device=q.device)
    if lse is None:
        lse = torch.empty(S["lse"], dtype=torch.float32, device=q.device)
    if idx is None:
        if p.flags & HILS_FLAG_GIVEN_IDX:
            raise ValueError("HILS_FLAG_GIVEN_IDX needs idx")
        idx = torch.empty(S["idx"], dtype=torch.int32, device=q.device)
    ws, n = _workspace(p, HILS_OP_DECODE, workspace)
    cp = p.c()
    _check(LIB.hils_decode_paged_fwd(
        ctypes.byref(cp), _ptr(q, "q", S["q"], dt), _ptr(k_pages, "k_pages", (P, p.Hkv, p.chunk, p.d), dt),
        _ptr(v_pages, "v_pages", (P, p.Hkv, p.chunk, p.d), dt), _ptr(lmk_pages, "lmk_pages", (P, Hl, p.d), dt),
        _ptr(bias_pages, "bias_pages", (P, Hl), torch.float32, False), _ptr(q_route, "q_route", S["q"], dt, False),
        _ptr(block_table, "block_table", (p.B, p.L // p.chunk), torch.int32), P,
        _ptr(seqlens, "seqlens", (p.B,), torch.int32, False), _ptr(out, "out", S["q"], dt),
        _ptr(lse, "lse", S["lse"], torch.float32), _ptr(idx, "idx", S["idx"], torch.int32),
        _ptr(ws, "workspace"), n, _stream()))
    return out, lse, idx


def hils_bwd(p: Params, dout, q, k, v, lmk, out, lse, idx, lmk_bias=None, q_route=None, want_dbias=True,
             workspace=None):
    """Backward with the selection fixed to ``idx``.  Returns dict(dq, dk, dv, dlmk, dlmk_bias, dq_route)."""
    S, dt = _shapes(p), p.torch_dtype
    dev = q.device
    dq = torch.empty(S["q"], dtype=dt, device=dev)
    dk = torch.empty(S["kv"], dtype=dt, device=dev)
    dv = torch.empty(S["kv"], dtype=dt, device=dev)
    dlmk = torch.empty(S["lmk"], dtype=dt, device=dev)
    dbias = torch.empty(S["bias"], dtype=torch.float32, device=dev) if want_dbias else None
    dqr = torch.empty(S["q"], dtype=dt, device=dev) if q_route is not None else None
    ws, n = _workspace(p, HILS_OP_BWD, workspace)
    cp = p.c()
    _check(LIB.hils_bwd(
        ctypes.byref(cp), _ptr(dout, "dout", S["q"], dt), _ptr(q, "q", S["q"], dt), _ptr(k, "k", S["kv"], dt),
        _ptr(v, "v", S["kv"], dt), _ptr(lmk, "lmk", S["lmk"], dt),
        _ptr(lmk_bias, "lmk_bias", S["bias"], torch.float32, False), _ptr(q_route, "q_route", S["q"], dt, False),
        _ptr(out, "out", S["q"], dt), _ptr(lse, "lse", S["lse"], torch.float32),
        _ptr(idx, "idx", S["idx"], torch.int32), _ptr(dq, "dq"), _ptr(dk, "dk"), _ptr(dv, "dv"),
        _ptr(dlmk, "dlmk"), _ptr(dbias, "dbias", required=False), _ptr(dqr, "dq_route", required=False),
        _ptr(ws, "workspace"), n, _stream()))
    return {"dq": dq, "dk": dk, "dv": dv, "dlmk": dlmk, "dlmk_bias": dbias, "dq_route": dqr}


def _lq_shape(p: Params, S):
    return (p.Hl or p.Hq, p.d) if p.flags & HILS_FLAG_SHARED_LMK_QUERY else S["lmk"]


def hils_landmark_fwd(p: Params, lq, k, lmk=None, lmk_bias=None):
    """Landmark compression (Prop. 3.1): lq [B, Hl, L/S, d] landmark queries (or
    [Hl, d] under HILS_FLAG_SHARED_LMK_QUERY) and k [B, Hkv, L, d] ->
    (lmk [B, Hl, L/S, d], lmk_bias [B, Hl, L/S] float32)."""
    S, dt = _shapes(p), p.torch_dtype
    dev = k.device
    lmk = torch.empty(S["lmk"], dtype=dt, device=dev) if lmk is None else lmk
    lmk_bias = torch.empty(S["bias"], dtype=torch.float32, device=dev) if lmk_bias is None else lmk_bias
    cp = p.c()
    _check(LIB.hils_landmark_fwd(ctypes.byref(cp), _ptr(lq, "lq", _lq_shape(p, S), dt), _ptr(k, "k", S["kv"], dt),
                                 _ptr(lmk, "lmk", S["lmk"], dt), _ptr(lmk_bias, "lmk_bias", S["bias"], torch.float32),
                                 _stream()))
    return lmk, lmk_bias


def hils_landmark_bwd(p: Params, lq, k, dlmk, dlmk_bias=None, dlq=None, dk=None, workspace=None):
    """Backward of hils_landmark_fwd -> (dlq [B, Hl, L/S, d] (or [Hl, d] under
    HILS_FLAG_SHARED_LMK_QUERY), dk [B, Hkv, L, d])."""
    S, dt = _shapes(p), p.torch_dtype
    dev = k.device
    lqs = _lq_shape(p, S)
    dlq = torch.empty(lqs, dtype=dt, device=dev) if dlq is None else dlq
    dk = torch.empty(S["kv"], dtype=dt, device=dev) if dk is None else dk
    ws, n = _workspace(p, HILS_OP_LANDMARK, workspace)
    cp = p.c()
    _check(LIB.hils_landmark_bwd(ctypes.byref(cp), _ptr(lq, "lq", lqs, dt), _ptr(k, "k", S["kv"], dt),
                                 _ptr(dlmk, "dlmk", S["lmk"], dt),
                                 _ptr(dlmk_bias, "dlmk_bias", S["bias"], torch.float32, False),
                                 _ptr(dlq, "dlq", lqs, dt), _ptr(dk, "dk", S["kv"], dt), _ptr(ws, "workspace"), n,
                                 _stream()))
    return dlq, dk


def hils_timing_enable(on: bool = True) -> None:
    """Bracket every library kernel launch of this thread with HIP events."""
    _check(LIB.hils_timing_enable(int(bool(on))))


def hils_timing_read(max_kernels: int = 64) -> dict:
    """Per kernel name: {"launches": n, "total_ms": t} for the launches recorded
    since timing was enabled (or last read); clears the records."""
    names = ctypes.create_string_buffer(4096)
    ms = (ctypes.c_float * max_kernels)()
    cnt = (ctypes.c_int * max_kernels)()
    nk = ctypes.c_int(0)
    _check(LIB.hils_timing_read(names, 4096, ms, cnt, max_kernels, ctypes.byref(nk)))
    keys = [k for k in names.value.decode().split("\n") if k]
    return {k: {"launches": cnt[i], "total_ms": ms[i]} for i, k in enumerate(keys[: nk.value])}
