"""Pins the vocabulary reference: a hand-worked example and the defining
properties (non-increasing ranked counts, ties by raw id, a bijection of the
kept words onto 0..V-1, the corpus rewritten through it)."""
import os

import numpy as np

import oracle
from paper_1611_06172_amd import inputs

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "vocab_example.txt")


def test_hand_worked_example():
    rows = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        key, *vals = line.split()
        rows[key] = [int(v) for v in vals]
    ranked, rank_of, V, corpus = oracle.build_vocab(rows["raw"], 8, rows["min_count"][0])
    assert V == rows["V"][0]
    assert ranked.tolist() == rows["ranked_counts"]
    assert rank_of.tolist() == rows["rank_of"]
    assert corpus.tolist() == rows["corpus"]


def test_properties_on_a_shuffled_zipf_stream():
    V_raw = 5000
    perm = np.random.default_rng(1).permutation(V_raw)
    raw = perm[inputs.zipf_ids(200_000, V_raw, 1.0, 2)].astype(np.int32)
    ranked, rank_of, V, corpus = oracle.build_vocab(raw, V_raw, 3)
    counts = np.bincount(raw, minlength=V_raw)
    assert V == int((counts >= 3).sum())
    assert np.all(np.diff(ranked[:V]) <= 0) and not ranked[V:].any()
    kept = np.flatnonzero(rank_of >= 0)
    assert sorted(rank_of[kept].tolist()) == list(range(V))
    assert np.array_equal(ranked[rank_of[kept]], counts[kept])
    # ties broken by increasing raw id
    by_rank = np.empty(V, np.int64)
    by_rank[rank_of[kept]] = kept
    same = ranked[1:V] == ranked[:V - 1]
    assert np.all(by_rank[1:V][same] > by_rank[:V - 1][same])
    assert np.array_equal(corpus, rank_of[raw])
