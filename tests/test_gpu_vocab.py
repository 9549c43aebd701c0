"""w2v_build_vocab against the vocabulary reference, bit for bit: ranked
counts, rank map, vocabulary size and the rewritten corpus; then a ranked
corpus trains through the atomic and split tiers."""
import numpy as np
import pytest

import oracle
from gpu_util import to_dev
from paper_1611_06172_amd import inputs, w2v

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("V_raw,T,min_count", [
    (8, 16, 2), (50_000, 1_000_000, 3), (1000, 0, 0), (300, 5000, 10_000), (1, 10, 0),
    (200_000, 5_000_001, 5),   # several 2^20-token chunks; tables overflow
    (30_000, 5_000_000, 0),    # one id range (bin) cut into several count units
    (4_194_304, 3_000_000, 1), # the largest vocabulary counted by bins: 128 bins
    (4_194_305, 1_000_000, 1), # one id more: the hash-table count
])
def test_vocab_matches_reference(V_raw, T, min_count):
    import torch
    if V_raw == 8:
        raw = np.array([3, 1, 3, 2, 3, 1, 7, 0, 5, 3, 1, 9, -1, 2, 6, 6], np.int32)
    else:
        perm = np.random.default_rng(V_raw).permutation(V_raw)
        raw = perm[inputs.zipf_ids(T, V_raw, 1.0, 3)].astype(np.int32)
        if T > 100:
            raw[::997] = V_raw + 5            # ids outside [0, V_raw)
            raw[5::1009] = -3
    ranked, rank_of, V, corpus = oracle.build_vocab(raw, V_raw, min_count)
    out = w2v.build_vocab(torch.from_numpy(raw).cuda(), V_raw, min_count)
    assert out["V"] == V
    assert np.array_equal(out["ranked_counts"].cpu().numpy(), ranked)
    assert np.array_equal(out["rank_of"].cpu().numpy(), rank_of)
    assert np.array_equal(out["corpus"].cpu().numpy(), corpus)


@pytest.mark.parametrize("kind", ["sorted", "constant", "two_bins_alternating"])
def test_vocab_unusual_streams(kind):
    """Streams whose ids are not spread over the chunks: sorted ids (each
    chunk holds one or two id ranges, so most segments are empty and a few
    fill whole chunks), one id repeated, and two ids from different ranges
    alternating; bit for bit against the reference."""
    import torch
    V_raw, T = 100_000, 3_000_017
    if kind == "sorted":
        raw = np.sort(inputs.zipf_ids(T, V_raw, 1.0, 8)).astype(np.int32)
    elif kind == "constant":
        raw = np.full(T, 65_537, np.int32)
    else:
        raw = np.where(np.arange(T) % 2 == 0, 7, 99_999).astype(np.int32)
    ranked, rank_of, V, corpus = oracle.build_vocab(raw, V_raw, 2)
    out = w2v.build_vocab(torch.from_numpy(raw).cuda(), V_raw, 2)
    assert out["V"] == V
    assert np.array_equal(out["ranked_counts"].cpu().numpy(), ranked)
    assert np.array_equal(out["rank_of"].cpu().numpy(), rank_of)
    assert np.array_equal(out["corpus"].cpu().numpy(), corpus)


def test_ranked_corpus_trains_with_update_tiers():
    """A shuffled-id stream ranked on the GPU: its tables, conflict-model
    thresholds and a concurrent epoch, against the serialised epoch of the
    same ranked corpus (loss within 2%)."""
    import torch
    V_raw = 20_000
    perm = np.random.default_rng(4).permutation(V_raw)
    raw = torch.from_numpy(perm[inputs.zipf_ids(400_000, V_raw, 1.0, 5)].astype(np.int32)).cuda()
    voc = w2v.build_vocab(raw, V_raw, min_count=2)
    V = voc["V"]
    counts = voc["ranked_counts"][:V].cpu().numpy()
    assert counts[0] == counts.max()
    table, thr = w2v.build_tables(counts, 0.75, 1e-3, 10**6)
    hot = w2v.hot_rows(counts, sample_t=1e-3, inflight=64)
    split = w2v.hot_rows(counts, sample_t=1e-3, inflight=64, tol=16.0)
    M0 = inputs.init_matrix(V, 64, "uniform", 6)
    losses = []
    for inflight, h, s in ((1, V, 0), (64, hot, split)):
        gi, go = to_dev(M0), torch.zeros((V, 64), device="cuda")
        lb = torch.zeros((1, 2), dtype=torch.float64, device="cuda")
        w2v.train_epoch(voc["corpus"], gi, go, to_dev(table),
                        torch.from_numpy(thr.view(np.int32)).cuda(), window=5, K=5,
                        seed=7, loss_buckets=lb, max_inflight=inflight, hot_rows=h,
                        split_rows=s)
        l = lb.cpu().numpy()
        losses.append(l[0, 0] / l[0, 1])
    assert abs(losses[1] - losses[0]) <= 0.02 * losses[0], losses
