"""Pins the oracle's HogBatch with negatives shared by groups of G
consecutive targets (the generalisation of Sec. 1.1's sharing):

  * G = 1 is the HogBatch epoch, bitwise;
  * one group's update is alpha times the negative gradient of the summed
    SGNS losses of its members, all at the rows as they were before the
    group (finite differences, numpy, independent of the oracle's code);
  * when every member's own negatives equal the shared ones (a one-word
    table), grouping departs from HogBatch only through the group snapshot,
    at second order in alpha.
"""
import math

import numpy as np
import pytest

import oracle
from paper_1611_06172_amd import inputs


def test_group_of_one_is_hogbatch():
    corpus = inputs.zipf_ids(20_000, 400, 1.0, 1)
    table, thr = oracle.build_tables(inputs.word_counts(corpus, 400), 0.75, 1e-3, 10**6)
    M_in = inputs.init_matrix(400, 24, "uniform", 2)
    M_out = inputs.init_matrix(400, 24, "normal", 3, scale=0.1)
    s = oracle.Sampling(corpus, table, thr, window=5, K=5, seed=4)
    a_in, a_out, h_in, h_out = M_in.copy(), M_out.copy(), M_in.copy(), M_out.copy()
    na, la = oracle.grouped_train_epoch(s, 1, a_in, a_out, n_buckets=3)
    nh, lh = oracle.train_epoch(s, h_in, h_out, n_buckets=3)
    assert na == nh
    assert np.array_equal(a_in.view(np.uint32), h_in.view(np.uint32))
    assert np.array_equal(a_out.view(np.uint32), h_out.view(np.uint32))
    np.testing.assert_array_equal(la, lh)


def group_loss(M_in, M_out, members, negs):
    total = 0.0
    for ctx, target in members:
        for c in ctx:
            a = M_in[c]
            total += math.log1p(math.exp(-float(a @ M_out[target])))
            for n in negs:
                if n != target:
                    total += math.log1p(math.exp(float(a @ M_out[n])))
    return total


@pytest.mark.parametrize("seed", [0, 1])
def test_one_group_is_alpha_times_negative_gradient(seed):
    """A single 7-token sentence, all its targets in one group of 8."""
    V, D, alpha = 10, 6, 0.05
    rng = np.random.default_rng(seed)
    corpus = rng.integers(0, V, 7).astype(np.int32)
    table = rng.integers(0, V, 1000).astype(np.int32)
    M_in = rng.normal(0, 0.5, (V, D)).astype(np.float32)
    M_out = rng.normal(0, 0.5, (V, D)).astype(np.float32)
    kw = dict(window=2, K=4, sentence_len=1000, seed=seed + 5, alpha0=alpha,
              min_alpha_frac=1.0)
    s = oracle.Sampling(corpus, table, None, **kw)
    mb = oracle.minibatches(s)
    members = [(list(c[c >= 0]), int(t)) for c, t in zip(mb["ctx"], mb["targets"])]
    negs = list(mb["negs"][0])            # drawn at the group's first position
    assert mb["pos"][0] == 0 and len(members) == 7
    g_in, g_out = M_in.copy(), M_out.copy()
    n, lb = oracle.grouped_train_epoch(s, 8, g_in, g_out, n_buckets=1)
    assert n == 7
    Mi, Mo = M_in.astype(np.float64), M_out.astype(np.float64)
    assert lb[0, 0] == pytest.approx(group_loss(Mi, Mo, members, negs), rel=1e-12)
    h = 1e-6
    for M, got in ((Mi, g_in), (Mo, g_out)):
        grad = np.zeros_like(M)
        for r in range(V):
            for j in range(D):
                old = M[r, j]
                M[r, j] = old + h
                lp = group_loss(Mi, Mo, members, negs)
                M[r, j] = old - h
                lm = group_loss(Mi, Mo, members, negs)
                M[r, j] = old
                grad[r, j] = (lp - lm) / (2 * h)
        before = M_in if M is Mi else M_out
        np.testing.assert_allclose(got.astype(np.float64) - before, -alpha * grad,
                                   rtol=1e-5, atol=2e-7)


def test_group_snapshot_departs_from_hogbatch_at_second_order():
    V, D = 60, 12
    corpus = inputs.zipf_ids(16, V - 1, 1.0, 13)   # short: no compounding
    table = np.full(1000, V - 1, np.int32)           # every negative is V-1
    M_in = inputs.init_matrix(V, D, "normal", 14, scale=0.3)
    M_out = inputs.init_matrix(V, D, "normal", 15, scale=0.3)
    diffs = []
    for alpha in (2e-3, 1e-3):
        kw = dict(window=3, K=3, seed=16, alpha0=alpha, min_alpha_frac=1.0)
        g_in, g_out, h_in, h_out = M_in.copy(), M_out.copy(), M_in.copy(), M_out.copy()
        oracle.grouped_train_epoch(oracle.Sampling(corpus, table, None, **kw), 4, g_in, g_out)
        oracle.train_epoch(oracle.Sampling(corpus, table, None, **kw), h_in, h_out)
        moved = np.abs(h_out.astype(np.float64) - M_out).max()
        diffs.append(max(np.abs(g_in.astype(np.float64) - h_in).max(),
                         np.abs(g_out.astype(np.float64) - h_out).max()))
        assert diffs[-1] < 0.05 * moved
    assert diffs[0] / diffs[1] == pytest.approx(4.0, rel=0.1)
