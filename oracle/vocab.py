"""Oracle: vocabulary of a raw id stream (count, rank by frequency, cut at a
minimum count). TEST INFRASTRUCTURE ONLY.

The paper trains on a counted corpus (Sec. 2); the plain definition is
written out with numpy: bincount for the counts and a stable sort for the
ranking (equal counts keep increasing raw id order)."""
import numpy as np


def build_vocab(raw, V_raw: int, min_count: int = 0):
    """Returns (ranked_counts int64[V_raw], rank_of int32[V_raw], V,
    corpus_out int32[T]) as w2v_build_vocab defines them."""
    raw = np.asarray(raw, dtype=np.int64)
    valid = (raw >= 0) & (raw < V_raw)
    counts = np.bincount(raw[valid], minlength=V_raw).astype(np.int64)
    order = np.argsort(-counts, kind="stable")
    kept = counts[order] >= max(int(min_count), 1)
    V = int(kept.sum())
    rank_of = np.full(V_raw, -1, np.int32)
    rank_of[order[:V]] = np.arange(V, dtype=np.int32)
    ranked = np.zeros(V_raw, np.int64)
    ranked[:V] = counts[order[:V]]
    corpus = np.full(raw.shape[0], -1, np.int32)
    corpus[valid] = rank_of[raw[valid]]
    return ranked, rank_of, V, corpus
