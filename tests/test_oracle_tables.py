"""Pins the oracle's sampling tables (negative table, subsampling thresholds).

Readings (the paper gives only "negative samples=5" and "sample=1e-4", Sec. 2,
and "sample one word from V", Alg. 1): negatives follow unigram^0.75; a word of
frequency f is kept with probability min(1, sqrt(t/f) + t/f). The pins below
check the table against the exact distribution it discretises and the
thresholds against values worked out by hand for frequencies that are powers
of two (so every intermediate is exact in binary).
"""
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def load_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append(line.split())
    return rows


def test_slot_counts_within_one_of_exact_share():
    rng = np.random.default_rng(3)
    counts = rng.integers(0, 10**6, size=5000).astype(np.int64)
    counts[::17] = 0
    size = 10**7
    table, _ = oracle.build_tables(counts, 0.75, 0.0, size, want_thresh=False)
    got = np.bincount(table, minlength=counts.size)
    q = counts.astype(np.float64) ** 0.75
    q /= q.sum()
    assert np.all(np.abs(got - size * q) <= 1.0 + 1e-6)
    assert np.all(got[counts == 0] == 0)
    assert np.all(np.diff(table) >= 0)          # ids in increasing order
    assert got.sum() == size


def test_uniform_counts_split_table_evenly():
    counts = np.full(8, 5, dtype=np.int64)
    table, _ = oracle.build_tables(counts, 0.75, 0.0, 64, want_thresh=False)
    assert table.tolist() == [w for w in range(8) for _ in range(8)]


def test_power_one_is_plain_unigram():
    counts = np.array([1, 3, 4], dtype=np.int64)   # shares 1/8, 3/8, 4/8
    table, _ = oracle.build_tables(counts, 1.0, 0.0, 16, want_thresh=False)
    assert np.bincount(table).tolist() == [2, 6, 8]


def test_keep_thresholds_hand_worked():
    """tests/golden/keep_thresholds.txt: t = 2^-13, total count 2^20."""
    rows = load_golden("keep_thresholds.txt")
    counts = np.array([int(r[0]) for r in rows], dtype=np.int64)
    filler = 2**20 - counts.sum()
    assert filler > 0
    counts_all = np.concatenate([counts, [filler]]).astype(np.int64)
    _, thr = oracle.build_tables(counts_all, 0.75, 2.0**-13, 16, want_table=False)
    for r, got in zip(rows, thr[:-1]):
        assert int(got) == int(r[1], 0), r


def test_no_subsampling_keeps_everything():
    counts = np.array([10**9, 1, 0, 5], dtype=np.int64)
    _, thr = oracle.build_tables(counts, 0.75, 0.0, 16, want_table=False)
    assert thr.tolist() == [0xFFFFFFFF] * 4


def test_keep_probability_matches_definition():
    """P(keep) = (thresh + 1) / 2^32 is within 2^-32 of min(1, sqrt(t/f)+t/f),
    and frequent words are kept no more often than rare ones."""
    rng = np.random.default_rng(4)
    counts = np.sort(rng.zipf(1.3, size=2000).astype(np.int64))[::-1].copy()
    t = 1e-4
    _, thr = oracle.build_tables(counts, 0.75, t, 16, want_table=False)
    f = counts / counts.sum()
    p = np.minimum(1.0, np.sqrt(t / f) + t / f)
    got = (thr.astype(np.float64) + 1.0) / 2**32
    assert np.all(np.abs(got - p) <= 2.0**-32 + 1e-15)
    assert np.all(np.diff(got) >= 0)            # counts are decreasing


def test_empirical_keep_rate():
    """Retained positions of the minibatch former follow the thresholds."""
    V = 4
    counts = np.array([2**16, 2**14, 2**12, 2**20 - 2**16 - 2**14 - 2**12],
                      dtype=np.int64)
    table, thr = oracle.build_tables(counts, 0.75, 2.0**-13, 64)
    p_keep = (thr.astype(np.float64) + 1) / 2**32
    n = 40000
    corpus = (np.arange(n) % V).astype(np.int32)     # position p holds p % V
    mb = oracle.minibatches(oracle.Sampling(corpus, table, thr, window=5, K=1,
                                            sentence_len=1000, seed=9))
    kept = np.bincount(corpus[mb["pos"]], minlength=V)
    total = np.bincount(corpus, minlength=V)
    for w in range(V):
        sd = math.sqrt(total[w] * p_keep[w] * (1 - p_keep[w]))
        assert abs(kept[w] - total[w] * p_keep[w]) <= 5 * sd + 1.0


def test_rejects_bad_arguments():
    with pytest.raises(ValueError):
        oracle.build_tables(np.array([-1, 2], dtype=np.int64))
    with pytest.raises(ValueError):
        oracle.build_tables(np.zeros(3, dtype=np.int64))
    with pytest.raises(ValueError):
        oracle.build_tables(np.ones(3, dtype=np.int64), table_size=2**32)
