"""The C-ABI boundary on the CPU: the library loads, exports every function
``include/hils.h`` declares, and rejects every invalid argument with its
documented code and a message before any HIP call (these run without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hils.h")
LIBPATH = os.path.join(ROOT, "paper_2607_02980_amd", "libhils.so")


@pytest.fixture(scope="module")
def hils():
    if not os.path.exists(LIBPATH):
        from paper_2607_02980_amd import build

        build.build()
    from paper_2607_02980_amd import hils as h

    return h


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hils_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(hils):
    names = declared_functions()
    assert {"hils_prefill_fwd", "hils_decode_fwd", "hils_bwd", "hils_workspace_size", "hils_last_error"} <= set(names)
    lib = ctypes.CDLL(LIBPATH)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in hils.h but not exported"
    assert hils.hils_version() >= 100


def params(hils, **kw):
    base = dict(B=1, Hq=8, Hkv=2, N=256, L=256, d=128, chunk=64, topk=8, window=128, dtype="bf16")
    base.update(kw)
    return hils.Params(**base)


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first


def call_prefill(hils, p, **override):
    ptrs = dict(q=FAKE, k=FAKE, v=FAKE, lmk=FAKE, bias=None, q_route=None, out=FAKE, lse=FAKE, idx=FAKE, ws=None)
    ptrs.update(override)
    cp = p.c()
    return hils.LIB.hils_prefill_fwd(ctypes.byref(cp), ptrs["q"], ptrs["k"], ptrs["v"], ptrs["lmk"], ptrs["bias"],
                                     ptrs["q_route"], ptrs["out"], ptrs["lse"], ptrs["idx"], ptrs["ws"], 0, None)


@pytest.mark.parametrize("kw,code,msg", [
    (dict(Hq=6, Hkv=4), 1, "multiple of Hkv"),
    (dict(Hl=4), 1, "Hl=4"),
    (dict(L=250, N=250), 1, "multiple of chunk"),
    (dict(N=512), 1, "N <= L"),
    (dict(topk=0), 1, ">= 1"),
    (dict(window=0), 1, ">= 1"),
    (dict(B=0), 1, ">= 1"),
    (dict(flags=16), 1, "unknown flags"),
    (dict(chunk=32), 2, "chunk 64"),
    (dict(d=96), 2, "d in {64, 128}"),
    (dict(Hq=6, Hkv=2), 2, "G=3"),
    (dict(Hq=32, Hkv=2), 2, "G=16"),
    (dict(topk=65), 2, "topk <= 64"),
])
def test_prefill_rejects_invalid_params(hils, kw, code, msg):
    rc = call_prefill(hils, params(hils, **kw))
    assert rc == code
    assert msg in hils.hils_last_error()


@pytest.mark.parametrize("name", ["q", "k", "v", "lmk", "out", "lse", "idx"])
def test_prefill_rejects_null_pointers(hils, name):
    rc = call_prefill(hils, params(hils), **{name: None})
    assert rc == hils.HILS_ERR_INVALID
    assert f"'{name}'" in hils.hils_last_error()


def test_params_null_and_bad_dtype_and_scale(hils):
    assert hils.LIB.hils_prefill_fwd(None, *([FAKE] * 4), None, None, FAKE, FAKE, FAKE, None, 0, None) == 1
    p = params(hils).c()
    p.dtype = 7
    n = ctypes.c_size_t()
    assert hils.LIB.hils_workspace_size(ctypes.byref(p), 0, ctypes.byref(n)) == 1
    p = params(hils).c()
    p.scale = float("inf")
    assert hils.LIB.hils_workspace_size(ctypes.byref(p), 0, ctypes.byref(n)) == 1
    assert "scale" in hils.hils_last_error()


def test_decode_needs_N_at_most_L(hils):
    p = params(hils, N=300, L=256).c()
    rc = hils.LIB.hils_decode_fwd(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, None, None, None, FAKE, FAKE, FAKE,
                                  None, 0, None)
    assert rc == hils.HILS_ERR_INVALID and "N <= L" in hils.hils_last_error()


def test_workspace_sizes_and_workspace_errors(hils):
    p = params(hils, B=2, N=1024, L=1024)
    assert hils.hils_workspace_size(p, hils.HILS_OP_PREFILL) >= 0
    need = hils.hils_workspace_size(p, hils.HILS_OP_BWD)
    nC = 1024 // 64
    assert need >= 4 * (2 * 2 * 1024 * 8 + 3 * 2 * 2 * nC)
    cp = p.c()
    args = [ctypes.byref(cp)] + [FAKE] * 5 + [None, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None]
    rc = hils.LIB.hils_bwd(*args, None, 0, None)
    assert rc == hils.HILS_ERR_WORKSPACE and "NULL" in hils.hils_last_error()
    rc = hils.LIB.hils_bwd(*args, FAKE, need - 1, None)
    assert rc == hils.HILS_ERR_WORKSPACE and f"{need} needed" in hils.hils_last_error()


def test_bwd_route_gradient_needs_its_buffer(hils):
    p = params(hils)
    cp = p.c()
    need = hils.hils_workspace_size(p, hils.HILS_OP_BWD)
    args = [ctypes.byref(cp), FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
            None, None, FAKE, need, None]
    assert hils.LIB.hils_bwd(*args) == hils.HILS_ERR_INVALID
    assert "dq_route" in hils.hils_last_error()


def test_bwd_rejects_forced_index_flag(hils):
    p = params(hils, flags=1)
    n = ctypes.c_size_t()
    cp = p.c()
    assert hils.LIB.hils_workspace_size(ctypes.byref(cp), 2, ctypes.byref(n)) == hils.HILS_ERR_INVALID


def test_binding_refuses_host_tensors(hils):
    import torch

    p = params(hils, dtype="f32", N=64, L=64)
    q = torch.zeros(1, 8, 64, 128)
    with pytest.raises(ValueError):
        hils._ptr(q, "q")


def test_error_string_is_thread_local(hils):
    import threading

    call_prefill(hils, params(hils, chunk=32))
    seen = {}

    def other():
        seen["msg"] = hils.hils_last_error()

    t = threading.Thread(target=other)
    t.start()
    t.join()
    assert seen["msg"] == ""
    assert "chunk" in hils.hils_last_error()


def test_timing_mode_without_launches(hils):
    hils.hils_timing_enable(True)
    assert hils.hils_timing_read() == {}
    hils.hils_timing_enable(False)


def test_landmark_entry_points_validate_on_the_host(hils):
    # N > L is fine for the compression (N is not used); no workspace is needed
    p = params(hils, N=4096, L=256)
    assert hils.hils_workspace_size(p, hils.HILS_OP_LANDMARK) == 0
    cp = p.c()
    assert hils.LIB.hils_landmark_fwd(ctypes.byref(cp), FAKE, FAKE, None, FAKE, None) == hils.HILS_ERR_INVALID
    assert "lmk" in hils.hils_last_error()
    assert hils.LIB.hils_landmark_fwd(ctypes.byref(cp), FAKE, FAKE, FAKE, None, None) == hils.HILS_ERR_INVALID
    assert "lmk_bias" in hils.hils_last_error()
    assert hils.LIB.hils_landmark_bwd(ctypes.byref(cp), FAKE, FAKE, FAKE, None, FAKE, None, None, 0, None) == \
        hils.HILS_ERR_INVALID
    assert "dk" in hils.hils_last_error()
    bad = params(hils, L=200).c()
    assert hils.LIB.hils_landmark_fwd(ctypes.byref(bad), FAKE, FAKE, FAKE, FAKE, None) == hils.HILS_ERR_INVALID
    assert "multiple of chunk" in hils.hils_last_error()
    odd = params(hils, d=96).c()
    assert hils.LIB.hils_landmark_bwd(ctypes.byref(odd), FAKE, FAKE, FAKE, None, FAKE, FAKE, None, 0, None) == \
        hils.HILS_ERR_UNSUPPORTED
    # the shared landmark query (one per head for every chunk) needs B*Hl*(L/S)*d floats
    # to sum its per-chunk gradients, and is a landmark-only flag
    sh = params(hils, B=2, Hq=8, Hkv=2, L=512, d=64, flags=hils.HILS_FLAG_SHARED_LMK_QUERY)
    assert hils.hils_workspace_size(sh, hils.HILS_OP_LANDMARK) == 2 * 8 * 8 * 64 * 4
    sc = sh.c()
    assert hils.LIB.hils_landmark_bwd(ctypes.byref(sc), FAKE, FAKE, FAKE, None, FAKE, FAKE, None, 0, None) == \
        hils.HILS_ERR_WORKSPACE
    assert hils.LIB.hils_landmark_bwd(ctypes.byref(sc), FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, 100, None) == \
        hils.HILS_ERR_WORKSPACE
    for op in (hils.HILS_OP_PREFILL, hils.HILS_OP_DECODE, hils.HILS_OP_BWD):
        with pytest.raises(hils.HilsError, match="landmark compression only"):
            hils.hils_workspace_size(params(hils, N=1, flags=hils.HILS_FLAG_SHARED_LMK_QUERY), op)
    gi = params(hils, flags=hils.HILS_FLAG_GIVEN_IDX).c()
    assert hils.LIB.hils_landmark_fwd(ctypes.byref(gi), FAKE, FAKE, FAKE, FAKE, None) == hils.HILS_ERR_INVALID


def test_paged_and_multi_token_decode_validate_on_the_host(hils):
    p1 = params(hils, B=4, N=1, L=4096, window=512)
    p4 = params(hils, B=4, N=4, L=4096, window=512)
    w1 = hils.hils_workspace_size(p1, hils.HILS_OP_DECODE)
    w4 = hils.hils_workspace_size(p4, hils.HILS_OP_DECODE)
    assert w4 > 3 * w1  # one set of records per (sequence, new query)
    with pytest.raises(hils.HilsError, match="N <= L"):
        hils.hils_workspace_size(params(hils, N=300, L=256), hils.HILS_OP_DECODE)
    with pytest.raises(hils.HilsError, match="B \\* N"):
        hils.hils_workspace_size(params(hils, B=300, N=256, L=256), hils.HILS_OP_DECODE)
    cp = p4.c()
    F = FAKE
    # (p, q, k_pages, v_pages, lmk_pages, bias_pages, q_route, block_table, num_pages, seqlens,
    #  out, lse, idx, workspace, ws_bytes, stream)
    rc = hils.LIB.hils_decode_paged_fwd(ctypes.byref(cp), F, F, F, F, None, None, None, 10, None, F, F, F, F, w4, None)
    assert rc == hils.HILS_ERR_INVALID and "block_table" in hils.hils_last_error()
    rc = hils.LIB.hils_decode_paged_fwd(ctypes.byref(cp), F, F, F, F, None, None, F, 0, None, F, F, F, F, w4, None)
    assert rc == hils.HILS_ERR_INVALID and "num_pages" in hils.hils_last_error()
    rc = hils.LIB.hils_decode_paged_fwd(ctypes.byref(cp), F, F, F, F, None, None, F, 10, None, F, F, F, F, w1, None)
    assert rc == hils.HILS_ERR_WORKSPACE


def test_head_normalised_selection_flag(hils):
    f = hils.HILS_FLAG_HEAD_NORM_SELECT
    assert hils.hils_workspace_size(params(hils, flags=f), hils.HILS_OP_PREFILL) >= 0
    assert hils.hils_workspace_size(params(hils, N=1, flags=f), hils.HILS_OP_DECODE) >= 0
    assert hils.hils_workspace_size(params(hils, flags=f), hils.HILS_OP_BWD) >= 0  # ignored there
    with pytest.raises(hils.HilsError, match="landmark compression"):
        hils.hils_workspace_size(params(hils, flags=f), hils.HILS_OP_LANDMARK)


def test_union_packing_needs_no_workspace(hils):
    # union packing keeps no per-slot records: its prefill workspace is 0, while
    # the chunk-major bf16 prefill reserves B*Hq*N*K*d bf16 partials (at least)
    f = hils.HILS_FLAG_UNION_PACKING
    p = params(hils, B=1, Hq=8, Hkv=2, N=1024, L=1024, d=128, topk=8)
    assert hils.hils_workspace_size(p, hils.HILS_OP_PREFILL) >= 8 * 1024 * 8 * 128 * 2
    pu = params(hils, B=1, Hq=8, Hkv=2, N=1024, L=1024, d=128, topk=8, flags=f)
    assert hils.hils_workspace_size(pu, hils.HILS_OP_PREFILL) == 0
    pg = params(hils, B=1, Hq=8, Hkv=2, N=1024, L=1024, d=128, topk=8, flags=f | hils.HILS_FLAG_GIVEN_IDX)
    assert hils.hils_workspace_size(pg, hils.HILS_OP_PREFILL) == 0


def test_noalloc_decode_rejects_calls_above_its_array(hils):
    # the no-allocation decode checks its workspace need against the fixed array
    # on the host, before any HIP call
    cap = hils.HILS_DECODE_NOALLOC_SCRATCH_BYTES
    small = params(hils, B=32, Hq=32, Hkv=8, N=1, L=131136, d=128, topk=16, window=512)
    assert hils.hils_workspace_size(small, hils.HILS_OP_DECODE) <= cap
    big = params(hils, B=256, Hq=32, Hkv=8, N=1, L=131136, d=128, topk=16, window=512)
    need = hils.hils_workspace_size(big, hils.HILS_OP_DECODE)
    assert need > cap
    cp = big.c()
    F = FAKE
    rc = hils.LIB.hils_decode_fwd_noalloc(ctypes.byref(cp), F, F, F, F, None, None, None, F, F, F, None)
    assert rc == hils.HILS_ERR_WORKSPACE
    assert f"{need} bytes" in hils.hils_last_error() and str(cap) in hils.hils_last_error()
    rc = hils.LIB.hils_decode_fwd_noalloc(ctypes.byref(small.c()), F, None, F, F, None, None, None, F, F, F, None)
    assert rc == hils.HILS_ERR_INVALID and "k_cache" in hils.hils_last_error()
    with open(HEADER) as f:
        assert f"HILS_DECODE_NOALLOC_SCRATCH_BYTES ((size_t){cap >> 20} << 20)" in f.read()


def test_prefill_record_cap_bounds_the_workspace(hils):
    # a long prefill runs its chunk-major passes over segments of rows whose
    # per-slot records fit the cap: the workspace shrinks with the cap, and bytes = 0
    # only reads it
    p = params(hils, B=1, Hq=32, Hkv=8, N=32768, L=32768, d=128, topk=16, window=512)
    full = hils.hils_workspace_size(p, hils.HILS_OP_PREFILL)
    per_row = 32 * 16 * (2 * 128 + 4)
    assert full >= 32768 * per_row
    old = hils.hils_prefill_record_cap(1 << 30)
    try:
        assert hils.hils_prefill_record_cap() == 1 << 30
        seg = hils.hils_workspace_size(p, hils.HILS_OP_PREFILL)
        # segments of the most whole 2048-row blocks that fit: 6144 rows, whose records
        # (plus the inverse index) make the workspace
        rows = (1 << 30) // per_row // 2048 * 2048
        assert rows == 6144
        assert rows * per_row <= seg < (rows + 2048) * per_row
        # a segment is at least 2048 rows, whatever the cap
        hils.hils_prefill_record_cap(1)
        tiny = hils.hils_workspace_size(p, hils.HILS_OP_PREFILL)
        assert 2048 * per_row <= tiny < seg
    finally:
        hils.hils_prefill_record_cap(old)
    assert hils.hils_workspace_size(p, hils.HILS_OP_PREFILL) == full
    # the default keeps the 512K-token prefill's workspace far below its 69 GB of records
    p512 = params(hils, B=1, Hq=32, Hkv=8, N=524288, L=524288, d=128, topk=16, window=512)
    assert hils.hils_workspace_size(p512, hils.HILS_OP_PREFILL) < 20e9 < 524288 * per_row
