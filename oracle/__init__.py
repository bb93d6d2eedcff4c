"""HiLS attention CPU oracle -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never loads it.

It wraps ``hils_oracle.c`` (a plain step-by-step statement of the paper's
forward, Sec. 2.1 and Eqs. (1), (9), (10), (11) with Appendix C's GQA
selection, and of the backward obtained by differentiating Eq. (10) with the
selection fixed).  The C file is compiled twice: ``f64`` (double arithmetic,
used for pins and parity) and ``f32`` (the plain fp32 variant).

Every array argument is a numpy array; inputs are float32 (bf16 data is
widened exactly), outputs are float64 (``f64``) or float32 (``f32``).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hils_oracle.c")
_LIBS = {"f64": os.path.join(_HERE, "liboracle_f64.so"), "f32": os.path.join(_HERE, "liboracle_f32.so")}
# HILS_ORACLE_SANITIZED=1 loads the AddressSanitizer/UBSan builds instead (build_sanitized;
# the process must preload clang's ASan runtime)
_SAN_LIBS = {k: v.replace(".so", "_san.so") for k, v in _LIBS.items()}
_CLANG = "/opt/rocm/llvm/bin/clang"


def build(verbose: bool = False) -> None:
    """Compile both precisions of the oracle with gcc + OpenMP."""
    for tag, real, isf in (("f64", "double", 0), ("f32", "float", 1)):
        out = _LIBS[tag]
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", f"-DREAL={real}",
               f"-DSUFFIX={tag}", f"-DREAL_IS_FLOAT={isf}", "-o", out + ".tmp", _SRC, "-lm"]
        if verbose:
            print(" ".join(cmd))
        subprocess.check_call(cmd)
        os.replace(out + ".tmp", out)


def build_sanitized(verbose: bool = False) -> None:
    """Both precisions compiled with clang under AddressSanitizer and
    UndefinedBehaviorSanitizer (single-threaded: no OpenMP), for the CPU
    sanitizer run of the pins."""
    for tag, real, isf in (("f64", "double", 0), ("f32", "float", 1)):
        out = _SAN_LIBS[tag]
        cmd = [_CLANG, "-O1", "-g", "-fPIC", "-shared", "-std=c11", "-fsanitize=address,undefined",
               "-fno-omit-frame-pointer", "-fno-sanitize-recover=undefined", f"-DREAL={real}",
               f"-DSUFFIX={tag}", f"-DREAL_IS_FLOAT={isf}", "-Wno-unknown-pragmas", "-o", out + ".tmp", _SRC, "-lm"]
        if verbose:
            print(" ".join(cmd))
        subprocess.check_call(cmd)
        os.replace(out + ".tmp", out)


class _Shape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int), ("Hq", ctypes.c_int), ("Hkv", ctypes.c_int), ("Hl", ctypes.c_int),
                ("N", ctypes.c_int), ("L", ctypes.c_int), ("d", ctypes.c_int), ("chunk", ctypes.c_int),
                ("topk", ctypes.c_int), ("window", ctypes.c_int), ("scale", ctypes.c_double),
                ("head_norm", ctypes.c_int)]


@dataclass
class Shape:
    B: int
    Hq: int
    Hkv: int
    Hl: int
    N: int
    L: int
    d: int
    chunk: int
    topk: int
    window: int
    scale: float
    head_norm: bool = False  # rank by per-head normalised scores (Sec. 4.1 variant)

    def c(self) -> _Shape:
        return _Shape(self.B, self.Hq, self.Hkv, self.Hl, self.N, self.L, self.d, self.chunk, self.topk,
                      self.window, float(self.scale), int(self.head_norm))


_loaded: dict[str, ctypes.CDLL] = {}


def _lib(prec: str) -> ctypes.CDLL:
    if prec not in _loaded:
        path = (_SAN_LIBS if os.environ.get("HILS_ORACLE_SANITIZED") == "1" else _LIBS)[prec]
        if not os.path.exists(path):
            build()
        _loaded[prec] = ctypes.CDLL(path)
    return _loaded[prec]


def _ptr(a):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data_as(ctypes.c_void_p)


def _f32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float32)


def _i32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.int32)


def _real(prec):
    return np.float64 if prec == "f64" else np.float32


def _check(shape: "Shape", **arrays):
    """Every array must have exactly the layout the C code indexes."""
    s = shape
    nc = s.L // s.chunk
    want = {"q": (s.B, s.Hq, s.N, s.d), "q_route": (s.B, s.Hq, s.N, s.d), "dout": (s.B, s.Hq, s.N, s.d),
            "k": (s.B, s.Hkv, s.L, s.d), "v": (s.B, s.Hkv, s.L, s.d), "lmk": (s.B, s.Hl, nc, s.d),
            "bias": (s.B, s.Hl, nc), "idx": (s.B, s.Hkv, s.N, s.topk), "qpos": (s.B, s.N)}
    for name, a in arrays.items():
        if a is not None and tuple(a.shape) != want[name]:
            raise ValueError(f"oracle: {name} has shape {tuple(a.shape)}, expected {want[name]}")


def fwd(shape: Shape, q, k, v, lmk, bias=None, q_route=None, qpos=None, rows=None, idx=None,
        prec: str = "f64", want_debug: bool = False):
    """Forward.  Returns dict(out, lse, idx[, sel_score, alpha]).

    If ``idx`` is given the selection is forced to it (forced-index mode);
    otherwise the oracle selects.  ``rows`` is an optional (n, 2) int array of
    (b, n) pairs; rows not listed are left as NaN (outputs) / -2 (idx).
    """
    lib = _lib(prec)
    R = _real(prec)
    s = shape
    q, k, v, lmk, bias, q_route = map(_f32, (q, k, v, lmk, bias, q_route))
    qpos = _i32(qpos)
    _check(s, q=q, k=k, v=v, lmk=lmk, bias=bias, q_route=q_route, qpos=qpos, idx=idx)
    rows_a = _i32(rows)
    nrows = 0 if rows_a is None else rows_a.shape[0]
    given = idx is not None
    idx_a = _i32(idx).copy() if given else np.full((s.B, s.Hkv, s.N, s.topk), -2, np.int32)
    out = np.full((s.B, s.Hq, s.N, s.d), np.nan, R)
    lse = np.full((s.B, s.Hq, s.N), np.nan, R)
    sel = np.full((s.B, s.Hq, s.N, s.topk), np.nan, R) if want_debug else None
    alpha = np.full((s.B, s.Hq, s.N, s.topk + 1), np.nan, R) if want_debug else None
    fn = getattr(lib, f"hils_oracle_fwd_{prec}")
    fn.restype = ctypes.c_int
    sh = s.c()
    rc = fn(ctypes.byref(sh), _ptr(q), _ptr(k), _ptr(v), _ptr(lmk), _ptr(bias), _ptr(q_route), _ptr(qpos),
            _ptr(rows_a), ctypes.c_int(nrows), ctypes.c_int(int(given)), _ptr(idx_a), _ptr(out), _ptr(lse),
            _ptr(sel), _ptr(alpha))
    if rc != 0:
        raise ValueError(f"oracle fwd failed with code {rc}")
    res = {"out": out, "lse": lse, "idx": idx_a}
    if want_debug:
        res["sel_score"] = sel
        res["alpha"] = alpha
    return res


def group_scores(shape: Shape, q, lmk, b, g, n, bias=None, q_route=None, qpos=None, prec: str = "f64"):
    """Group scores sigma_c (max over the group's heads of the surrogate score)
    of query (b, n) for KV group g, over its candidate chunks."""
    lib = _lib(prec)
    R = _real(prec)
    q, lmk, bias, q_route = map(_f32, (q, lmk, bias, q_route))
    qpos = _i32(qpos)
    _check(shape, q=q, lmk=lmk, bias=bias, q_route=q_route, qpos=qpos)
    sigma = np.zeros(shape.L // shape.chunk, R)
    fn = getattr(lib, f"hils_oracle_group_scores_{prec}")
    fn.restype = ctypes.c_long
    sh = shape.c()
    nc = fn(ctypes.byref(sh), _ptr(q), _ptr(lmk), _ptr(bias), _ptr(q_route), _ptr(qpos), ctypes.c_int(b),
            ctypes.c_int(g), ctypes.c_int(n), _ptr(sigma))
    if nc < 0:
        raise ValueError("oracle group_scores failed")
    return sigma[:nc].copy()


def dense_weights(shape: Shape, q, k, lmk, idx, bias=None, q_route=None, qpos=None, prec: str = "f64"):
    """Dense per-head weight matrix w[B, Hq, N, L] from Appendix C's case-wise definition."""
    lib = _lib(prec)
    R = _real(prec)
    q, k, lmk, bias, q_route = map(_f32, (q, k, lmk, bias, q_route))
    idx = _i32(idx)
    qpos = _i32(qpos)
    _check(shape, q=q, k=k, lmk=lmk, bias=bias, q_route=q_route, qpos=qpos, idx=idx)
    w = np.zeros((shape.B, shape.Hq, shape.N, shape.L), R)
    fn = getattr(lib, f"hils_oracle_dense_weights_{prec}")
    fn.restype = ctypes.c_int
    sh = shape.c()
    rc = fn(ctypes.byref(sh), _ptr(q), _ptr(k), _ptr(lmk), _ptr(bias), _ptr(q_route), _ptr(qpos), _ptr(idx),
            _ptr(w))
    if rc:
        raise ValueError("oracle dense_weights failed")
    return w


def bwd(shape: Shape, dout, q, k, v, lmk, idx, bias=None, q_route=None, qpos=None, rows=None,
        prec: str = "f64", want_dbias: bool = True, only_group: int = -1):
    """Backward with the selection fixed to ``idx``.  Returns dict(dq, dk, dv,
    dlmk, dbias, dq_route); ``dq_route`` is None (folded into dq) unless a
    routing query is given.  With ``rows`` only those rows contribute; with
    ``only_group`` >= 0 only that KV group's gradients are computed."""
    lib = _lib(prec)
    R = _real(prec)
    s = shape
    dout, q, k, v, lmk, bias, q_route = map(_f32, (dout, q, k, v, lmk, bias, q_route))
    idx = _i32(idx)
    qpos = _i32(qpos)
    _check(s, dout=dout, q=q, k=k, v=v, lmk=lmk, bias=bias, q_route=q_route, qpos=qpos, idx=idx)
    rows_a = _i32(rows)
    nrows = 0 if rows_a is None else rows_a.shape[0]
    nc = s.L // s.chunk
    dq = np.zeros((s.B, s.Hq, s.N, s.d), R)
    dk = np.zeros((s.B, s.Hkv, s.L, s.d), R)
    dv = np.zeros((s.B, s.Hkv, s.L, s.d), R)
    dlmk = np.zeros((s.B, s.Hl, nc, s.d), R)
    dbias = np.zeros((s.B, s.Hl, nc), R) if want_dbias else None
    dqr = np.zeros((s.B, s.Hq, s.N, s.d), R) if q_route is not None else None
    fn = getattr(lib, f"hils_oracle_bwd_{prec}")
    fn.restype = ctypes.c_int
    sh = s.c()
    rc = fn(ctypes.byref(sh), _ptr(dout), _ptr(q), _ptr(k), _ptr(v), _ptr(lmk), _ptr(bias), _ptr(q_route),
            _ptr(qpos), _ptr(rows_a), ctypes.c_int(nrows), _ptr(idx), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dlmk),
            _ptr(dbias), _ptr(dqr), ctypes.c_int(only_group))
    if rc:
        raise ValueError(f"oracle bwd failed with code {rc}")
    return {"dq": dq, "dk": dk, "dv": dv, "dlmk": dlmk, "dbias": dbias, "dq_route": dqr}


def _shared_query(s: Shape, lq):
    """The landmark-token-free variant (Sec. 4.1): one learnable query per
    landmark head, [Hl, d], used as q'_c for every chunk of every sequence."""
    lq = np.asarray(lq, np.float32)
    if lq.shape != (s.Hl, s.d):
        raise ValueError(f"shared landmark query: expected [{s.Hl}, {s.d}], got {list(lq.shape)}")
    return np.ascontiguousarray(np.broadcast_to(lq[None, :, None, :], (s.B, s.Hl, s.L // s.chunk, s.d)))


def landmark_fwd(shape: Shape, lq, k, prec: str = "f64", shared: bool = False):
    """Landmark compression (Prop. 3.1): lq [B, Hl, L/S, d] landmark queries q'_c
    (or [Hl, d] with shared=True: one query per head for all chunks), k [B, Hkv, L, d].
    Returns dict(lmk = k'_c [B, Hl, L/S, d], bias = b'_c [B, Hl, L/S])."""
    lib = _lib(prec)
    R = _real(prec)
    s = shape
    if shared:
        lq = _shared_query(s, lq)
    lq, k = _f32(lq), _f32(k)
    _check(s, lmk=lq, k=k)
    nc = s.L // s.chunk
    lmk = np.zeros((s.B, s.Hl, nc, s.d), R)
    bias = np.zeros((s.B, s.Hl, nc), R)
    fn = getattr(lib, f"hils_oracle_landmark_fwd_{prec}")
    fn.restype = ctypes.c_int
    sh = s.c()
    if fn(ctypes.byref(sh), _ptr(lq), _ptr(k), _ptr(lmk), _ptr(bias)):
        raise ValueError("oracle landmark_fwd failed")
    return {"lmk": lmk, "bias": bias}


def landmark_bwd(shape: Shape, lq, k, dlmk, dbias=None, prec: str = "f64", shared: bool = False):
    """Backward of the landmark compression for upstream dlmk (of k'_c) and
    dbias (of b'_c, None = 0).  Returns dict(dlq [B, Hl, L/S, d], dk [B, Hkv, L, d]).
    With shared=True lq is [Hl, d] and dlq [Hl, d] is the sum of the per-chunk
    gradients over every chunk and sequence that used the shared query."""
    lib = _lib(prec)
    R = _real(prec)
    s = shape
    if shared:
        lq = _shared_query(s, lq)
    lq, k, dlmk, dbias = _f32(lq), _f32(k), _f32(dlmk), _f32(dbias)
    _check(s, lmk=lq, k=k, bias=dbias)
    _check(s, lmk=dlmk)
    nc = s.L // s.chunk
    dlq = np.zeros((s.B, s.Hl, nc, s.d), R)
    dk = np.zeros((s.B, s.Hkv, s.L, s.d), R)
    fn = getattr(lib, f"hils_oracle_landmark_bwd_{prec}")
    fn.restype = ctypes.c_int
    sh = s.c()
    if fn(ctypes.byref(sh), _ptr(lq), _ptr(k), _ptr(dlmk), _ptr(dbias), _ptr(dlq), _ptr(dk)):
        raise ValueError("oracle landmark_bwd failed")
    if shared:
        dlq = dlq.sum(axis=(0, 2))
    return {"dlq": dlq, "dk": dk}


def decode_positions(shape: Shape, seqlens=None):
    """Positions [B, N] of the N new queries of each sequence in a decode step:
    the N tokens that end the sequence (their k/v already in the cache), query n
    of sequence b at len_b - N + n with len_b = seqlens[b] clamped into [N, L]
    (None: L).  N = 1 is plain decode; N > 1 verifies N drafted tokens at once,
    each attending causally up to its own position."""
    s = shape
    lens = np.full(s.B, s.L, np.int64) if seqlens is None else np.clip(np.asarray(seqlens, np.int64), s.N, s.L)
    return (lens[:, None] - s.N + np.arange(s.N)[None, :]).astype(np.int32)


def gather_pages(shape: Shape, block_table, k_pages, v_pages, lmk_pages, bias_pages=None):
    """Per-sequence caches from a paged pool in which a page holds one chunk:
    chunk c of sequence b is page block_table[b, c].  Pools: k/v [P, Hkv, S, d],
    landmarks [P, Hl, d], bias [P, Hl].  Returns dense (k, v, lmk, bias) in the
    [B, Hkv, L, d] / [B, Hl, L/S, d] / [B, Hl, L/S] layouts of fwd()."""
    s = shape
    nc = s.L // s.chunk
    t = np.asarray(block_table, np.int64)
    if t.shape != (s.B, nc):
        raise ValueError(f"block_table has shape {t.shape}, expected {(s.B, nc)}")
    # [B, nc, Hkv, S, d] -> [B, Hkv, nc, S, d] -> [B, Hkv, L, d]
    k = np.asarray(k_pages)[t].transpose(0, 2, 1, 3, 4).reshape(s.B, s.Hkv, s.L, s.d)
    v = np.asarray(v_pages)[t].transpose(0, 2, 1, 3, 4).reshape(s.B, s.Hkv, s.L, s.d)
    lmk = np.asarray(lmk_pages)[t].transpose(0, 2, 1, 3)
    bias = None if bias_pages is None else np.asarray(bias_pages)[t].transpose(0, 2, 1)
    return (np.ascontiguousarray(k), np.ascontiguousarray(v), np.ascontiguousarray(lmk),
            None if bias is None else np.ascontiguousarray(bias))


def decode(shape: Shape, q, k, v, lmk, seqlens=None, bias=None, q_route=None, idx=None, rows=None,
           prec: str = "f64", block_table=None):
    """Decode step of N >= 1 new queries per sequence (q [B, Hq, N, d]) against
    caches, contiguous ([B, Hkv, L, d], ...) or, with block_table, paged pools
    (see gather_pages).  Returns fwd()'s dict."""
    if block_table is not None:
        k, v, lmk, bias = gather_pages(shape, block_table, k, v, lmk, bias)
    return fwd(shape, q, k, v, lmk, bias=bias, q_route=q_route, qpos=decode_positions(shape, seqlens), rows=rows,
               idx=idx, prec=prec)


def chunk_overlap(idx, M: int) -> float:
    """Normalised chunk-overlap ratio of blocks of M adjacent queries (the
    measure of the kernel-design section, Sec. 4.2): (M K - |union of their top-K
    sets|) / ((M - 1) K), averaged over every block of M consecutive rows (per
    sequence and KV group) whose rows all hold K valid entries.  1 means the M
    queries retrieve the same chunks, 0 that they share none.  idx [B, Hkv, N, K]."""
    idx = np.asarray(idx)
    B, Hkv, N, K = idx.shape
    vals = []
    for b in range(B):
        for g in range(Hkv):
            for n0 in range(0, N - M + 1, M):
                blk = idx[b, g, n0:n0 + M]
                if (blk < 0).any():
                    continue
                u = len(np.unique(blk))
                vals.append((M * K - u) / ((M - 1) * K))
    return float(np.mean(vals)) if vals else float("nan")


def n_candidates(i: int, chunk: int, window: int) -> int:
    """|C_i| = l(i)/S with l(i) clamped at 0 (Sec. 2.1)."""
    return max(0, (i - window + 1) // chunk)


class swapped_library:
    """Context manager: route calls of precision ``prec`` to another build of the
    oracle source (the mutation tests plant a mistake in a copy and check that
    the pins catch it)."""

    def __init__(self, path: str, prec: str = "f64"):
        self.path, self.prec = path, prec

    def __enter__(self):
        self.saved = _loaded.get(self.prec)
        _loaded[self.prec] = ctypes.CDLL(self.path)
        return self

    def __exit__(self, *exc):
        if self.saved is None:
            _loaded.pop(self.prec, None)
        else:
            _loaded[self.prec] = self.saved
        return False


def build_variant(src_text: str, out_path: str) -> str:
    """Compile an edited copy of the oracle source (f64) to ``out_path``."""
    src = out_path + ".c"
    with open(src, "w") as f:
        f.write(src_text)
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-DREAL=double",
                           "-DSUFFIX=f64", "-DREAL_IS_FLOAT=0", "-o", out_path, src, "-lm"])
    return out_path
