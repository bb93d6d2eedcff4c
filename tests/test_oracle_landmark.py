"""Pins of the oracle's landmark compression (Prop. 3.1): k'_c is the attention
of the landmark query q'_c over its chunk's keys and b'_c the entropy of that
attention.

Each pin reaches the oracle's output by a route other than its own code:
  * Prop. 3.1 is exact at the Taylor point: scale q'.k' + b' equals the
    log-sum-exp of the chunk's logits (scipy's logsumexp), and the gradient of
    that log-sum-exp at q' (central differences) is scale * k'.
  * b' lies in [0, log S]; q' = 0 gives b' = log S and k' = the mean key; one
    dominant logit gives b' -> 0 and k' -> that key (the two regimes named next
    to the proposition).
  * S = 2 reduces to a logistic split: scipy's expit and entropy.
  * The backward matches central finite differences of a scalar loss in fp64,
    and differentiating the Taylor-point identity (which holds for every q')
    gives a null direction: upstream gradients (scale q', 1) give dq' = 0.
  * Hl = Hq sums each group's heads into dk: it equals the heads run one by one.
"""
import math

import numpy as np
import pytest
from scipy.special import expit, logsumexp
from scipy.stats import entropy

import oracle

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def shape(B=1, Hq=4, Hkv=2, Hl=None, L=256, d=16, S=64, scale=None):
    return oracle.Shape(B=B, Hq=Hq, Hkv=Hkv, Hl=Hl or Hq, N=1, L=L, d=d, chunk=S, topk=1, window=1,
                        scale=scale if scale is not None else 1.0 / math.sqrt(d))


def rand(rng, *shp, sd=1.0):
    return (rng.standard_normal(shp) * sd).astype(np.float32)


def group_of(s, hl):
    return hl // (s.Hl // s.Hkv)


def chunk_keys(s, k, b, hl, c):
    g = group_of(s, hl)
    return k[b, g, c * s.chunk:(c + 1) * s.chunk].astype(np.float64)


@pytest.mark.parametrize("Hl_eq_Hq", [True, False])
def test_taylor_point_identity_and_gradient(Hl_eq_Hq):
    rng = np.random.default_rng(11)
    s = shape(Hl=None if Hl_eq_Hq else 2)
    nc = s.L // s.chunk
    lq = rand(rng, s.B, s.Hl, nc, s.d, sd=2.0)
    k = rand(rng, s.B, s.Hkv, s.L, s.d)
    r = oracle.landmark_fwd(s, lq, k)
    for hl in range(s.Hl):
        for c in range(nc):
            K = chunk_keys(s, k, 0, hl, c)
            qc = lq[0, hl, c].astype(np.float64)
            f = lambda q: logsumexp(s.scale * K @ q)
            # Prop. 3.1 holds with equality at q = q'_c
            assert abs(s.scale * qc @ r["lmk"][0, hl, c] + r["bias"][0, hl, c] - f(qc)) < 1e-12
            # and its linear term is the gradient there: grad f(q'_c) = scale * k'_c
            h = 1e-6
            grad = np.array([(f(qc + h * e) - f(qc - h * e)) / (2 * h) for e in np.eye(s.d)])
            np.testing.assert_allclose(grad, s.scale * r["lmk"][0, hl, c], rtol=0, atol=1e-7)


def test_entropy_range_and_uniform_regime():
    rng = np.random.default_rng(12)
    s = shape()
    nc = s.L // s.chunk
    k = rand(rng, s.B, s.Hkv, s.L, s.d)
    lq = rand(rng, s.B, s.Hl, nc, s.d, sd=3.0)
    r = oracle.landmark_fwd(s, lq, k)
    assert (r["bias"] >= -1e-12).all() and (r["bias"] <= math.log(s.chunk) + 1e-12).all()
    # q' = 0: uniform attention, b' = log S, k' = the chunk's mean key
    r0 = oracle.landmark_fwd(s, np.zeros_like(lq), k)
    np.testing.assert_allclose(r0["bias"], math.log(s.chunk), rtol=0, atol=1e-12)
    for hl in range(s.Hl):
        for c in range(nc):
            np.testing.assert_allclose(r0["lmk"][0, hl, c], chunk_keys(s, k, 0, hl, c).mean(0), rtol=0, atol=1e-12)


def test_dominant_logit_regime():
    # keys: key 5 of every chunk points along e_0, the others are orthogonal to it
    s = shape(Hq=2, Hkv=1, L=128, d=8, scale=1.0)
    nc = s.L // s.chunk
    rng = np.random.default_rng(13)
    k = np.zeros((1, 1, s.L, s.d), np.float32)
    k[..., 1:] = rand(rng, 1, 1, s.L, s.d - 1)
    k[0, 0, 5::s.chunk, 0] = 1.0
    k[0, 0, 5::s.chunk, 1:] = 0.0
    lq = np.zeros((1, s.Hl, nc, s.d), np.float32)
    lq[..., 0] = 60.0
    r = oracle.landmark_fwd(s, lq, k)
    assert (r["bias"] < 1e-20).all()
    for c in range(nc):
        np.testing.assert_allclose(r["lmk"][0, :, c], np.broadcast_to(k[0, 0, c * s.chunk + 5], (s.Hl, s.d)),
                                   rtol=0, atol=1e-20)


def test_two_key_chunks_reduce_to_a_logistic_split():
    rng = np.random.default_rng(14)
    s = shape(Hq=2, Hkv=2, L=8, d=4, S=2)
    nc = s.L // s.chunk
    k = rand(rng, s.B, s.Hkv, s.L, s.d)
    lq = rand(rng, s.B, s.Hl, nc, s.d, sd=2.0)
    r = oracle.landmark_fwd(s, lq, k)
    for hl in range(s.Hl):
        for c in range(nc):
            K = chunk_keys(s, k, 0, hl, c)
            z = s.scale * K @ lq[0, hl, c].astype(np.float64)
            p1 = expit(z[1] - z[0])
            assert abs(r["bias"][0, hl, c] - entropy([1 - p1, p1])) < 1e-12
            np.testing.assert_allclose(r["lmk"][0, hl, c], (1 - p1) * K[0] + p1 * K[1], rtol=0, atol=1e-12)


def _loss(s, lq, k, dl, db):
    r = oracle.landmark_fwd(s, lq, k)
    return float((r["lmk"] * dl).sum() + (r["bias"] * db).sum())


@pytest.mark.parametrize("Hl_eq_Hq,with_bias", [(True, True), (False, True), (True, False)])
def test_backward_matches_finite_differences(Hl_eq_Hq, with_bias):
    # inputs on a dyadic grid, so the perturbed float32 inputs are exact
    rng = np.random.default_rng(15)
    s = shape(Hq=4, Hkv=2, Hl=None if Hl_eq_Hq else 2, L=128, d=8)
    nc = s.L // s.chunk
    q = lambda *shp: np.round(rand(rng, *shp) * 64) / 64
    lq, k = q(s.B, s.Hl, nc, s.d), q(s.B, s.Hkv, s.L, s.d)
    dl = rand(rng, s.B, s.Hl, nc, s.d).astype(np.float64)
    db = rand(rng, s.B, s.Hl, nc).astype(np.float64) if with_bias else np.zeros((s.B, s.Hl, nc))
    g = oracle.landmark_bwd(s, lq, k, dl, db if with_bias else None)
    h = 2.0 ** -12
    for name, arr, grad in (("lq", lq, g["dlq"]), ("k", k, g["dk"])):
        for flat in rng.choice(arr.size, 24, replace=False):
            i = np.unravel_index(flat, arr.shape)
            xp, xm = arr.copy(), arr.copy()
            xp[i] += h
            xm[i] -= h
            args_p = (xp, k) if name == "lq" else (lq, xp)
            args_m = (xm, k) if name == "lq" else (lq, xm)
            fd = (_loss(s, *args_p, dl, db) - _loss(s, *args_m, dl, db)) / (2 * h)
            assert abs(fd - grad[i]) < 1e-5 * max(1.0, abs(fd)), (name, i, fd, grad[i])


def test_taylor_identity_gives_a_null_direction():
    # f(q') = scale q'.k'(q') + b'(q') for every q'; differentiating, the upstream
    # gradients (dk', db') = (scale q', 1) give dq' = scale k' - scale k' = 0
    rng = np.random.default_rng(16)
    s = shape(L=192, d=16)
    nc = s.L // s.chunk
    lq = rand(rng, s.B, s.Hl, nc, s.d, sd=2.0)
    k = rand(rng, s.B, s.Hkv, s.L, s.d)
    g = oracle.landmark_bwd(s, lq, k, s.scale * lq.astype(np.float64), np.ones((s.B, s.Hl, nc)))
    np.testing.assert_allclose(g["dlq"], 0.0, rtol=0, atol=1e-12)


def test_group_heads_sum_into_dk():
    rng = np.random.default_rng(17)
    s = shape(Hq=4, Hkv=2, L=128, d=8)
    nc = s.L // s.chunk
    lq = rand(rng, s.B, s.Hl, nc, s.d)
    k = rand(rng, s.B, s.Hkv, s.L, s.d)
    dl = rand(rng, s.B, s.Hl, nc, s.d)
    db = rand(rng, s.B, s.Hl, nc)
    g = oracle.landmark_bwd(s, lq, k, dl, db)
    one = shape(Hq=1, Hkv=1, L=128, d=8)
    dk = np.zeros_like(g["dk"])
    for hl in range(s.Hl):
        gg = group_of(s, hl)
        r = oracle.landmark_bwd(one, lq[:, hl:hl + 1], k[:, gg:gg + 1], dl[:, hl:hl + 1], db[:, hl:hl + 1])
        dk[:, gg] += r["dk"][:, 0]
        np.testing.assert_allclose(g["dlq"][:, hl], r["dlq"][:, 0], rtol=0, atol=1e-12)
    np.testing.assert_allclose(g["dk"], dk, rtol=0, atol=1e-12)


def test_shared_query_variant_matches_finite_differences():
    # Sec. 4.1's landmark-token-free variant: one query per landmark head for every
    # chunk; its gradient is checked by central differences of the loss in that query
    rng = np.random.default_rng(18)
    s = shape(B=2, Hq=4, Hkv=2, L=192, d=8)
    nc = s.L // s.chunk
    q = lambda *shp: np.round(rand(rng, *shp) * 64) / 64
    lq, k = q(s.Hl, s.d), q(s.B, s.Hkv, s.L, s.d)
    dl = rand(rng, s.B, s.Hl, nc, s.d).astype(np.float64)
    db = rand(rng, s.B, s.Hl, nc).astype(np.float64)
    r = oracle.landmark_fwd(s, lq, k, shared=True)
    # forward: every chunk sees the same query, so chunk c of head hl matches the
    # per-chunk attention of that one query (scipy's logsumexp route of Prop. 3.1)
    for b in range(s.B):
        for hl in range(s.Hl):
            for c in range(nc):
                K = chunk_keys(s, k, b, hl, c)
                assert abs(s.scale * lq[hl].astype(np.float64) @ r["lmk"][b, hl, c] + r["bias"][b, hl, c]
                           - logsumexp(s.scale * K @ lq[hl].astype(np.float64))) < 1e-12
    g = oracle.landmark_bwd(s, lq, k, dl, db, shared=True)
    assert g["dlq"].shape == (s.Hl, s.d)

    def loss(x):
        rr = oracle.landmark_fwd(s, x, k, shared=True)
        return float((rr["lmk"] * dl).sum() + (rr["bias"] * db).sum())

    h = 2.0 ** -12
    for hl in range(s.Hl):
        for dd in range(s.d):
            xp, xm = lq.copy(), lq.copy()
            xp[hl, dd] += h
            xm[hl, dd] -= h
            fd = (loss(xp) - loss(xm)) / (2 * h)
            assert abs(fd - g["dlq"][hl, dd]) < 1e-5 * max(1.0, abs(fd)), (hl, dd, fd, g["dlq"][hl, dd])
    # dk is the per-chunk backward's dk with the broadcast query
    full = oracle.landmark_bwd(s, np.broadcast_to(lq[None, :, None], (s.B, s.Hl, nc, s.d)), k, dl, db)
    np.testing.assert_array_equal(g["dk"], full["dk"])
