"""GPU minibatch formation equals the oracle's bit for bit.

w2v_debug_minibatches runs the epoch kernel's own sampling code (subsampling,
compaction, window shrink, shared negatives, masks, learning rates) and writes
the minibatches out; every field must equal oracle.minibatches exactly.
"""
import numpy as np
import pytest

import oracle
from paper_1611_06172_amd import inputs, w2v
from gpu_util import assert_same_minibatches, expect_device_flag, gpu_minibatches, thresh_dev, to_dev

pytestmark = pytest.mark.gpu


def run_both(corpus, V, table, thr, **kw):
    o = oracle.minibatches(oracle.Sampling(corpus, table, thr, **kw))
    g = w2v.debug_minibatches(to_dev(corpus), to_dev(table), thresh_dev(thr), V=V, **kw)
    import torch
    torch.cuda.synchronize()
    return gpu_minibatches(g, kw.get("pos_begin", 0)), o


CASES = [
    # V, T, s, sample_t, window, K, L, epoch, n_epochs, seed, table_size
    (1000, 200_000, 1.0, 0.0, 5, 5, 1000, 0, 1, 7, 10**8),     # tiny config, full
    (1000, 50_000, 1.0, 1e-3, 5, 5, 1000, 0, 1, 8, 10**6),     # with subsampling
    (5000, 40_000, 1.1, 1e-3, 8, 25, 1000, 3, 5, 9, 10**7),    # window 8, K 25, epoch 3
    (300, 30_007, 1.0, 1e-2, 16, 64, 1024, 1, 2, 10, 99_991),  # max window/K/sentence, ragged
    (50, 3_001, 1.0, 0.0, 1, 0, 7, 0, 1, 11, 64),              # K = 0, tiny sentences
]


@pytest.mark.parametrize("case", CASES)
def test_minibatches_bitwise(case):
    V, T, s, t, w, K, L, e, E, seed, tsize = case
    corpus = inputs.zipf_ids(T, V, s, seed)
    table, thr = oracle.build_tables(inputs.word_counts(corpus, V), 0.75, t, tsize)
    if t == 0.0:
        thr = None
    g, o = run_both(corpus, V, table, thr, window=w, K=K, sentence_len=L,
                    epoch=e, n_epochs=E, seed=seed * 1000 + 1)
    assert len(o["targets"]) > 0 or K == 0
    assert_same_minibatches(g, o)


def test_sub_range():
    V, T = 800, 60_000
    corpus = inputs.zipf_ids(T, V, 1.0, 12)
    table, thr = oracle.build_tables(inputs.word_counts(corpus, V), 0.75, 1e-3, 10**6)
    g, o = run_both(corpus, V, table, thr, window=5, K=5, sentence_len=1000,
                    pos_begin=17_000, pos_end=41_000, seed=5)
    assert_same_minibatches(g, o)


def test_large_vocab_prefix():
    """The throughput workload's shapes: V = 1e6 Zipf(1.07), t = 1e-4, a 1e8
    slot table, first 2e5 tokens."""
    V = 1_000_000
    corpus = inputs.zipf_ids(200_000, V, 1.07, 6)
    counts = np.rint(inputs.zipf_pmf(V, 1.07) * 1e9).astype(np.int64)
    table, thr = oracle.build_tables(counts, 0.75, 1e-4, 10**8)
    g, o = run_both(corpus, V, table, thr, window=5, K=5, sentence_len=1000, seed=6)
    kept = len(o["targets"]) / 200_000
    assert 0.4 < kept < 0.7
    assert_same_minibatches(g, o)


def test_rejects_out_of_range_corpus_ids():
    import torch
    V = 100
    corpus = inputs.zipf_ids(5000, V, 1.0, 13)
    corpus[100] = V
    corpus[2000] = -5
    table, _ = oracle.build_tables(inputs.word_counts(np.clip(corpus, 0, V - 1), V),
                                   0.75, 0.0, 1000)
    stats = torch.zeros(5, dtype=torch.int64, device="cuda")
    out = w2v.debug_minibatches(to_dev(corpus), to_dev(table), None, V=V,
                                window=3, K=2, sentence_len=500, stats=stats)
    torch.cuda.synchronize()
    t = out["targets"].cpu().numpy()
    assert t[100] == -1 and t[2000] == -1
    assert stats[3].item() == 2 and stats[2].item() == 5000
    expect_device_flag()
