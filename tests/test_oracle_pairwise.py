"""Pins the oracle's Algorithm 1 (per-pair Hogwild SGD, the paper's
baseline) against facts that do not depend on its own code:

  * sampling: input word 0 draws exactly the negatives a HogBatch minibatch
    shares, and every input word's private draws follow the table;
  * with one input word per target and distinct output words, Algorithm 1
    and the HogBatch step are the same computation, so the two oracle epochs
    agree to rounding (the HogBatch step is pinned by finite differences);
  * with several input words per target (or repeated negatives) Algorithm 1
    moves the shared target row between input words and departs from the
    HogBatch step at second order in alpha;
  * rows of words that never occur stay bitwise unchanged; training lowers
    the loss.
"""
import numpy as np
import pytest

import oracle
from paper_1611_06172_amd import inputs


def small_config(V=300, T=6000, seed=1, D=16):
    corpus = inputs.zipf_ids(T, V, 1.0, seed)
    table, _ = oracle.build_tables(inputs.word_counts(corpus, V), 0.75, 0.0, 10**6,
                                   want_thresh=False)
    M_in = inputs.init_matrix(V, D, "uniform", seed + 1)
    M_out = inputs.init_matrix(V, D, "normal", seed + 2, scale=0.1)
    return corpus, table, M_in, M_out


def test_input_word_0_draws_the_shared_negatives():
    corpus, table, _, _ = small_config()
    s = oracle.Sampling(corpus, table, None, window=5, K=5, sentence_len=1000, seed=4)
    mb = oracle.minibatches(s)
    for m in range(0, len(mb["targets"]), 97):
        neg = oracle.pair_negatives(s, int(mb["pos"][m]), 3)
        assert np.array_equal(neg[0], mb["negs"][m])


def test_private_negatives_follow_table_distribution():
    V = 20
    counts = (1000 // np.arange(1, V + 1)).astype(np.int64)
    table, _ = oracle.build_tables(counts, 0.75, 0.0, 10**6, want_thresh=False)
    q = counts ** 0.75 / (counts ** 0.75).sum()
    s = oracle.Sampling(np.zeros(4000, np.int32), table, None, window=5, K=4, seed=6)
    draws = np.concatenate([oracle.pair_negatives(s, p, 10)[1:].ravel()
                            for p in range(0, 4000, 4)])
    hist = np.bincount(draws, minlength=V)
    exp = q * draws.size
    chi2 = ((hist - exp) ** 2 / exp).sum()
    assert chi2 < 43.8  # 19 dof, p = 1e-3


def test_one_input_word_and_distinct_outputs_equals_hogbatch():
    """Two-token sentences give every target exactly one input word; a table
    holding only a word that never occurs makes the one negative distinct
    from every target."""
    V, D = 50, 12
    corpus = inputs.zipf_ids(4000, V - 1, 1.0, 9)          # ids < V-1
    table = np.full(1000, V - 1, np.int32)
    M_in = inputs.init_matrix(V, D, "uniform", 10)
    M_out = inputs.init_matrix(V, D, "normal", 11, scale=0.2)
    kw = dict(window=3, K=1, sentence_len=2, seed=12, alpha0=0.05)
    a_in, a_out = M_in.copy(), M_out.copy()
    h_in, h_out = M_in.copy(), M_out.copy()
    na, la = oracle.pairwise_train_epoch(oracle.Sampling(corpus, table, None, **kw),
                                         a_in, a_out, n_buckets=2)
    nh, lh = oracle.train_epoch(oracle.Sampling(corpus, table, None, **kw),
                                h_in, h_out, n_buckets=2)
    assert na == nh == len(corpus)
    np.testing.assert_allclose(a_in, h_in, rtol=0, atol=1e-7)
    np.testing.assert_allclose(a_out, h_out, rtol=0, atol=1e-7)
    np.testing.assert_allclose(la, lh, rtol=1e-12)


@pytest.mark.parametrize("sentence_len,K", [(1000, 3), (2, 2)])
def test_departs_from_hogbatch_at_second_order(sentence_len, K):
    """Several input words share the target row (long sentences), or one
    input word meets a repeated negative (K = 2): the per-pair order matters
    only at second order in alpha. A one-word table makes every private
    negative the shared one (otherwise the two methods draw different
    negatives and differ at first order)."""
    V, D = 60, 12
    corpus = inputs.zipf_ids(16, V - 1, 1.0, 13)   # short: no compounding
    table = np.full(1000, V - 1, np.int32)
    M_in = inputs.init_matrix(V, D, "normal", 14, scale=0.3)
    M_out = inputs.init_matrix(V, D, "normal", 15, scale=0.3)
    diffs = []
    for alpha in (2e-3, 1e-3):
        kw = dict(window=3, K=K, sentence_len=sentence_len, seed=16, alpha0=alpha,
                  min_alpha_frac=1.0)
        a_in, a_out = M_in.copy(), M_out.copy()
        h_in, h_out = M_in.copy(), M_out.copy()
        oracle.pairwise_train_epoch(oracle.Sampling(corpus, table, None, **kw), a_in, a_out)
        oracle.train_epoch(oracle.Sampling(corpus, table, None, **kw), h_in, h_out)
        moved = np.abs(h_out.astype(np.float64) - M_out).max()
        diffs.append(max(np.abs(a_in.astype(np.float64) - h_in).max(),
                         np.abs(a_out.astype(np.float64) - h_out).max()))
        assert diffs[-1] < 0.05 * moved
    assert diffs[0] / diffs[1] == pytest.approx(4.0, rel=0.1)


def test_untouched_rows_and_training_lowers_loss():
    V, D = 400, 16
    corpus = inputs.zipf_ids(20_000, 200, 1.0, 17)          # ids < 200
    table, _ = oracle.build_tables(inputs.word_counts(corpus, V), 0.75, 0.0, 10**6,
                                   want_thresh=False)
    M_in = inputs.init_matrix(V, D, "uniform", 18)
    M_out = np.zeros((V, D), np.float32)
    a_in, a_out = M_in.copy(), M_out.copy()
    losses = []
    for e in range(3):
        s = oracle.Sampling(corpus, table, None, window=5, K=5, seed=19, epoch=e, n_epochs=3)
        _, b = oracle.pairwise_train_epoch(s, a_in, a_out, n_buckets=1)
        losses.append(b[0, 0] / b[0, 1])
    assert losses[1] < losses[0] and losses[2] < losses[0]
    assert np.array_equal(a_in[200:].view(np.uint32), M_in[200:].view(np.uint32))
    assert not a_out[200:].any()


def test_matches_an_independent_per_pair_restatement():
    """Alg. 1 restated independently in numpy from the per-pair logistic
    step (for each input word in window order: the target pair, then that
    word's own draws, a draw equal to the target forming no pair; each pair
    reads its output row as the earlier pairs left it and writes it back at
    once; the input row moves by the sum of its pairs' steps after its last
    pair), on the minibatches and private draws of the oracle's sampling
    (pinned elsewhere). A three-word table makes private draws repeat within
    one input word's K and across input words, and hit the target. The two
    agree to within one fp32 rounding per write of the row (fp64 inner
    products summed in another order)."""
    V, D = 12, 8
    corpus = np.array([0, 3, 1, 4, 2, 5, 0, 6, 1, 7, 2, 8, 0, 9, 1, 10, 2, 11, 3, 4,
                       5, 6, 0, 1, 2, 7, 8, 9, 10, 11, 0, 2, 4, 6, 8, 10, 1, 3, 5, 7],
                      np.int32)
    table = np.array([0] * 5 + [1] * 3 + [2] * 2, np.int32)
    M_in = inputs.init_matrix(V, D, "normal", 20, scale=0.4)
    M_out = inputs.init_matrix(V, D, "normal", 21, scale=0.4)
    kw = dict(window=3, K=3, sentence_len=len(corpus), seed=22, alpha0=0.1)
    s = oracle.Sampling(corpus, table, None, **kw)
    mb = oracle.minibatches(s)

    r_in, r_out = M_in.astype(np.float32).copy(), M_out.astype(np.float32).copy()
    writes_in, writes_out = np.zeros(V, int), np.zeros(V, int)
    saw_repeat = saw_hit = saw_three = False
    for m in range(len(mb["targets"])):
        t, a = int(mb["targets"][m]), float(mb["alpha"][m])
        inputs_m = [int(c) for c in mb["ctx"][m] if c >= 0]
        draws = oracle.pair_negatives(s, int(mb["pos"][m]), len(inputs_m))
        saw_three |= len(inputs_m) >= 3
        for i, c in enumerate(inputs_m):
            saw_repeat |= len(set(draws[i].tolist())) < kw["K"]
            saw_hit |= bool((draws[i] == t).any())
            pairs = [(t, 1.0)] + [(int(w), 0.0) for w in draws[i] if w != t]
            v = r_in[c].astype(np.float64)
            step = np.zeros(D)
            for w, label in pairs:
                u = r_out[w].astype(np.float64)
                g = a * (label - 1.0 / (1.0 + np.exp(-float(np.dot(v, u)))))
                step += g * u
                r_out[w] = (u + g * v).astype(np.float32)
                writes_out[w] += 1
            r_in[c] = (v + step).astype(np.float32)
            writes_in[c] += 1
    assert saw_repeat and saw_hit and saw_three

    o_in, o_out = M_in.copy(), M_out.copy()
    n, _ = oracle.pairwise_train_epoch(s, o_in, o_out)
    assert n == len(mb["targets"])
    for got, ref, writes in ((o_in, r_in, writes_in), (o_out, r_out, writes_out)):
        ulp = np.spacing(np.maximum(np.abs(got), np.abs(ref)).astype(np.float32))
        bound = np.maximum(writes, 1)[:, None] * ulp
        assert np.all(np.abs(got.astype(np.float64) - ref) <= bound), \
            np.max(np.abs(got.astype(np.float64) - ref) / ulp)
    assert writes_in.sum() >= 3 and writes_out.max() >= 3
