"""Pins of the per-head normalised selection (the wording of Sec. 4.1: each
query head's chunk weights are normalised before the maximum over the group's
heads), a variant of the ranking of App. C.  The normalised group score is
max_h (s^_hc - log sum_{c' in C_i} exp(s^_hc')).

  * A worked example computed by hand: a head with uniformly high scores loses
    to a head with one decisive chunk once both are normalised (the raw maximum
    picks the other chunk).
  * With one head per group (MHA) normalising subtracts a per-row constant: the
    selection equals the raw one.
  * Invariance: shifting all of one head's scores by a constant (through its
    landmark bias) changes the raw selection but not the normalised one.
"""
import math

import numpy as np
import pytest

import oracle


def shape(**kw):
    base = dict(B=1, Hq=2, Hkv=1, Hl=2, N=5, L=5, d=1, chunk=1, topk=1, window=1, scale=1.0)
    base.update(kw)
    return oracle.Shape(**base)


def test_hand_worked_example():
    # q = 0, so s^_hc = b'_hc exactly.  Query 4 (S = 1, W = 1) has candidates 0..3.
    # head 0: 5.0, 4.9, 4.8, 4.7 -> log-weights -1.2425, -1.3425, -1.4425, -1.5425
    #   (log-sum-exp 5 + log(1 + e^-0.1 + e^-0.2 + e^-0.3) = 6.2425)
    # head 1: 0, 0, 3, 0 -> log-weights -3.1392, -3.1392, -0.1392, -3.1392
    #   (log-sum-exp log(3 + e^3) = 3.1392)
    # raw max: 5.0, 4.9, 4.8, 4.7 -> chunk 0; normalised max: chunk 2
    bias = np.zeros((1, 2, 5), np.float32)
    bias[0, 0, :4] = [5.0, 4.9, 4.8, 4.7]
    bias[0, 1, :4] = [0.0, 0.0, 3.0, 0.0]
    z = np.zeros((1, 2, 5, 1), np.float32)
    kv = np.ones((1, 1, 5, 1), np.float32)
    lmk = np.zeros((1, 2, 5, 1), np.float32)
    raw = oracle.fwd(shape(), z, kv, kv, lmk, bias=bias)
    nrm = oracle.fwd(shape(head_norm=True), z, kv, kv, lmk, bias=bias)
    assert raw["idx"][0, 0, 4, 0] == 0
    assert nrm["idx"][0, 0, 4, 0] == 2
    sig = oracle.group_scores(shape(head_norm=True), z, lmk, 0, 0, 4, bias=bias)
    np.testing.assert_allclose(sig, [-1.2425, -1.3425, -0.1392, -1.5425], atol=1e-4)
    lse0 = 5 + math.log(1 + math.exp(-0.1) + math.exp(-0.2) + math.exp(-0.3))
    assert abs(sig[0] - (5.0 - lse0)) < 1e-6


def rand_case(rng, s, with_bias=True):
    nc = s.L // s.chunk
    q = rng.standard_normal((s.B, s.Hq, s.N, s.d)).astype(np.float32)
    k = rng.standard_normal((s.B, s.Hkv, s.L, s.d)).astype(np.float32)
    v = rng.standard_normal((s.B, s.Hkv, s.L, s.d)).astype(np.float32)
    lmk = rng.standard_normal((s.B, s.Hl, nc, s.d)).astype(np.float32)
    bias = (0.5 * rng.standard_normal((s.B, s.Hl, nc))).astype(np.float32) if with_bias else None
    return q, k, v, lmk, bias


def test_one_head_per_group_keeps_the_raw_selection():
    rng = np.random.default_rng(31)
    s = shape(B=2, Hq=4, Hkv=4, Hl=4, N=300, L=320, d=16, chunk=16, topk=5, window=40, scale=0.3)
    q, k, v, lmk, bias = rand_case(rng, s)
    raw = oracle.fwd(s, q, k, v, lmk, bias=bias)
    s.head_norm = True
    nrm = oracle.fwd(s, q, k, v, lmk, bias=bias)
    np.testing.assert_array_equal(raw["idx"], nrm["idx"])
    np.testing.assert_array_equal(raw["out"], nrm["out"])


def test_a_shift_of_one_heads_scores_changes_only_the_raw_selection():
    rng = np.random.default_rng(32)
    s = shape(B=1, Hq=4, Hkv=1, Hl=4, N=400, L=448, d=16, chunk=16, topk=4, window=40, scale=0.3)
    q, k, v, lmk, bias = rand_case(rng, s)
    shifted = bias.copy()
    shifted[:, 1] += 3.0   # head 1's scores all up by 3
    shifted[:, 2] -= 2.0   # head 2's all down by 2
    raw_a = oracle.fwd(s, q, k, v, lmk, bias=bias)["idx"]
    raw_b = oracle.fwd(s, q, k, v, lmk, bias=shifted)["idx"]
    assert (raw_a != raw_b).any()  # the raw maximum follows the shifted head
    s.head_norm = True
    nrm_a = oracle.fwd(s, q, k, v, lmk, bias=bias)["idx"]
    nrm_b = oracle.fwd(s, q, k, v, lmk, bias=shifted)["idx"]
    np.testing.assert_array_equal(nrm_a, nrm_b)
    assert (nrm_a != raw_a).any()  # and normalising does change the ranking
