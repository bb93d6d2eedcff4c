"""Pins of the oracle's decode step for the paged cache and for N new queries per
sequence (speculative verification), the two pieces the decode oracle adds to
fwd(): page gathering and query positions.

  * Paging: an identity page table over a pool that is the contiguous cache cut
    into chunks gives bit-identical results; so does any permutation of the
    pool's pages with the table permuted alike, a pool with unused pages, and
    sequences that share their first pages (the contiguous caches then hold the
    shared chunks twice).
  * Multi-token: query n of an N-token step at length len equals a one-token
    step at length len - N + n + 1; N tokens at len = L are the last N rows of
    the prefill of the same sequence; with the exact-mass construction (keys
    constant inside a chunk, landmark = that key, bias log S) and K >= |C_i|,
    the N-token step is textbook causal attention at those positions.
  * Lengths are clamped into [N, L].
"""
import numpy as np
import pytest

import oracle
from tests.oracle_helpers import dense_causal, p2_construction


def rnd(rng, *shape):
    return rng.standard_normal(shape).astype(np.float32)


def shape(B=3, Hq=4, Hkv=2, Hl=None, N=1, L=256, d=16, S=16, K=3, W=20, scale=0.35):
    return oracle.Shape(B=B, Hq=Hq, Hkv=Hkv, Hl=Hl or Hq, N=N, L=L, d=d, chunk=S, topk=K, window=W, scale=scale)


def caches(rng, s, bias=True):
    nc = s.L // s.chunk
    k, v = rnd(rng, s.B, s.Hkv, s.L, s.d), rnd(rng, s.B, s.Hkv, s.L, s.d)
    lmk = rnd(rng, s.B, s.Hl, nc, s.d)
    b = rnd(rng, s.B, s.Hl, nc) if bias else None
    return k, v, lmk, b


def to_pages(s, k, v, lmk, bias):
    """The contiguous caches cut into one-chunk pages, page b * nc + c."""
    nc = s.L // s.chunk
    kp = k.reshape(s.B, s.Hkv, nc, s.chunk, s.d).transpose(0, 2, 1, 3, 4).reshape(s.B * nc, s.Hkv, s.chunk, s.d)
    vp = v.reshape(s.B, s.Hkv, nc, s.chunk, s.d).transpose(0, 2, 1, 3, 4).reshape(s.B * nc, s.Hkv, s.chunk, s.d)
    lp = lmk.transpose(0, 2, 1, 3).reshape(s.B * nc, s.Hl, s.d)
    bp = None if bias is None else bias.transpose(0, 2, 1).reshape(s.B * nc, s.Hl)
    table = np.arange(s.B * nc, dtype=np.int32).reshape(s.B, nc)
    return kp, vp, lp, bp, table


def same(a, b):
    for key in ("out", "lse", "idx"):
        np.testing.assert_array_equal(a[key], b[key], err_msg=key)


@pytest.mark.parametrize("N", [1, 3])
def test_identity_paging_equals_contiguous_cache(N):
    rng = np.random.default_rng(21)
    s = shape(N=N)
    k, v, lmk, bias = caches(rng, s)
    q = rnd(rng, s.B, s.Hq, N, s.d)
    lens = [256, 97, 40]
    ref = oracle.decode(s, q, k, v, lmk, seqlens=lens, bias=bias)
    kp, vp, lp, bp, table = to_pages(s, k, v, lmk, bias)
    same(oracle.decode(s, q, kp, vp, lp, seqlens=lens, bias=bp, block_table=table), ref)


def test_permuted_pool_with_unused_pages_and_a_shared_prefix():
    rng = np.random.default_rng(22)
    s = shape(N=2)
    nc = s.L // s.chunk
    k, v, lmk, bias = caches(rng, s)
    # sequence 2 shares the first 5 chunks of sequence 0 (a common prompt prefix)
    k[2, :, :5 * s.chunk], v[2, :, :5 * s.chunk] = k[0, :, :5 * s.chunk], v[0, :, :5 * s.chunk]
    lmk[2, :, :5], bias[2, :, :5] = lmk[0, :, :5], bias[0, :, :5]
    q = rnd(rng, s.B, s.Hq, s.N, s.d)
    lens = [200, 256, 150]
    ref = oracle.decode(s, q, k, v, lmk, seqlens=lens, bias=bias)
    kp, vp, lp, bp, table = to_pages(s, k, v, lmk, bias)
    table[2, :5] = table[0, :5]  # the copies in sequence 2's own pages become unused
    P = s.B * nc + 7             # plus 7 pages that no table names
    perm = rng.permutation(P)    # page p of the ordered pool is stored at perm[p]
    pools = []
    for x in (kp, vp, lp, bp):
        y = rnd(rng, P, *x.shape[1:])
        y[perm[: x.shape[0]]] = x
        pools.append(y)
    same(oracle.decode(s, q, *pools[:3], seqlens=lens, bias=pools[3], block_table=perm[table]), ref)


def test_token_n_of_a_multi_token_step_is_a_single_token_step():
    rng = np.random.default_rng(23)
    N = 5
    s = shape(N=N, K=4, W=33)
    k, v, lmk, bias = caches(rng, s)
    q = rnd(rng, s.B, s.Hq, N, s.d)
    lens = [256, 130, 70]
    r = oracle.decode(s, q, k, v, lmk, seqlens=lens, bias=bias)
    one = shape(N=1, K=4, W=33)
    for n in range(N):
        r1 = oracle.decode(one, q[:, :, n:n + 1], k, v, lmk, seqlens=[x - N + n + 1 for x in lens], bias=bias)
        np.testing.assert_array_equal(r["out"][:, :, n:n + 1], r1["out"])
        np.testing.assert_array_equal(r["lse"][:, :, n:n + 1], r1["lse"])
        np.testing.assert_array_equal(r["idx"][:, :, n:n + 1], r1["idx"])


def test_multi_token_step_at_full_length_is_the_end_of_the_prefill():
    rng = np.random.default_rng(24)
    N, L = 6, 192
    pre = shape(B=2, N=L, L=L, K=3, W=40)
    k, v, lmk, bias = caches(rng, pre)
    q = rnd(rng, pre.B, pre.Hq, L, pre.d)
    ref = oracle.fwd(pre, q, k, v, lmk, bias=bias)
    s = shape(B=2, N=N, L=L, K=3, W=40)
    r = oracle.decode(s, np.ascontiguousarray(q[:, :, L - N:]), k, v, lmk, bias=bias)
    np.testing.assert_array_equal(r["out"], ref["out"][:, :, L - N:])
    np.testing.assert_array_equal(r["lse"], ref["lse"][:, :, L - N:])
    np.testing.assert_array_equal(r["idx"], ref["idx"][:, :, L - N:])


@pytest.mark.parametrize("paged", [False, True])
def test_exact_mass_multi_token_step_is_dense_causal(paged):
    rng = np.random.default_rng(25)
    B, Hq, Hkv, Hl, S, L, d, N = 2, 4, 2, 4, 8, 128, 8, 4
    _, k, lmk, bias = p2_construction(rng, B, Hq, Hkv, Hl, L, d, S)
    v = rnd(rng, B, Hkv, L, d)
    q = rnd(rng, B, Hq, N, d)
    s = shape(B=B, Hq=Hq, Hkv=Hkv, Hl=Hl, N=N, L=L, d=d, S=S, K=L // S, W=9, scale=0.5)
    lens = [128, 77]
    if paged:
        kp, vp, lp, bp, table = to_pages(s, k, v, lmk, bias)
        r = oracle.decode(s, q, kp, vp, lp, seqlens=lens, bias=bp, block_table=table)
    else:
        r = oracle.decode(s, q, k, v, lmk, seqlens=lens, bias=bias)
    qpos = np.array([[n + x - N for n in range(N)] for x in lens])
    ref, ref_lse = dense_causal(q, k, v, 0.5, qpos=qpos)
    np.testing.assert_allclose(r["out"], ref, atol=2e-7, rtol=0)
    np.testing.assert_allclose(r["lse"], ref_lse, atol=2e-7, rtol=0)


def test_lengths_are_clamped_into_N_to_L():
    s = shape(B=4, N=3, L=64)
    pos = oracle.decode_positions(s, [0, 2, 3, 1000])
    np.testing.assert_array_equal(pos, [[0, 1, 2], [0, 1, 2], [0, 1, 2], [61, 62, 63]])
    np.testing.assert_array_equal(oracle.decode_positions(s), [[61, 62, 63]] * 4)


def test_chunk_overlap_measure():
    # the overlap ratio of the kernel-design section: identical sets -> 1, disjoint -> 0,
    # and a hand-computed block: M = 2, K = 3, sets {1, 2, 3} and {2, 3, 7}: union 4,
    # (6 - 4) / 3 = 2/3
    same = np.tile(np.array([[1, 2, 3]]), (4, 1))[None, None]
    assert oracle.chunk_overlap(same, 4) == 1.0
    disjoint = np.arange(12).reshape(4, 3)[None, None]
    assert oracle.chunk_overlap(disjoint, 4) == 0.0
    ex = np.array([[1, 2, 3], [2, 3, 7]])[None, None]
    assert abs(oracle.chunk_overlap(ex, 2) - 2 / 3) < 1e-12
    # blocks with padded (-1) entries are skipped
    pad = np.array([[1, 2, -1], [1, 2, 3]])[None, None]
    assert np.isnan(oracle.chunk_overlap(pad, 2))
