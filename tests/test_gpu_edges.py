"""Edge cases of the epoch through the C ABI: maximal shapes, degenerate
corpora and ranges, and what the kernels must leave untouched."""
import numpy as np
import pytest

import oracle
from gpu_util import expect_device_flag, thresh_dev, to_dev
from paper_1611_06172_amd import inputs, w2v
from test_gpu_train_epoch import gpu_epoch, rel_row_error

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("algorithm,D,window", [
    ("hogbatch", 640, 5),     # ten columns per lane, K+1 = 65 in 11 blocks of 6
    ("hogbatch", 128, 16),    # up to 32 input words, 33 blocks of 2
    ("pairwise", 640, 16)])   # per input word: any window at any D
def test_maximal_shapes(algorithm, D, window):
    """The largest compiled shapes: K = 64, 1024-token sentences, D up to
    640, window up to 16 (HogBatch keeps all N rows in registers, so window
    16 is compiled up to D = 128)."""
    V = 700
    corpus = inputs.zipf_ids(6000, V, 1.0, 31)
    table, _ = oracle.build_tables(inputs.word_counts(corpus, V), 0.75, 0.0, 10**6,
                                   want_thresh=False)
    M_in = inputs.init_matrix(V, D, "uniform", 32)
    M_out = inputs.init_matrix(V, D, "normal", 33, scale=0.02)
    kw = dict(window=window, K=64, sentence_len=1024, seed=34)
    o_in, o_out = M_in.copy(), M_out.copy()
    run = oracle.pairwise_train_epoch if algorithm == "pairwise" else oracle.train_epoch
    n, _ = run(oracle.Sampling(corpus, table, None, **kw), o_in, o_out)
    gi, go, stats, _ = gpu_epoch(corpus, table, None, M_in, M_out, max_inflight=1,
                                 algorithm=algorithm, **kw)
    assert stats[0] == n
    assert rel_row_error(gi, o_in) < 2e-4
    assert rel_row_error(go, o_out) < 2e-4


def test_uncompiled_shape_is_reported():
    import torch
    c = torch.zeros(2000, dtype=torch.int32, device="cuda")
    M = torch.zeros((10, 640), device="cuda")
    tb = torch.zeros(4, dtype=torch.int32, device="cuda")
    with pytest.raises(w2v.W2VError) as err:
        w2v.train_epoch(c, M, M.clone(), tb, window=16, K=5)
    assert err.value.code == w2v.EUNSUPPORTED


@pytest.mark.parametrize("algorithm", ["hogbatch", "pairwise"])
def test_degenerate_corpora(algorithm):
    """A one-token corpus, an empty range, a corpus whose every position is
    subsampled away, and one-token sentences form no minibatch and leave the
    matrices bitwise unchanged; raw positions are still counted."""
    import torch
    V, D = 50, 32
    table = np.arange(V, dtype=np.int32)
    M_in = inputs.init_matrix(V, D, "uniform", 35)
    M_out = inputs.init_matrix(V, D, "normal", 36, scale=0.1)
    cases = [
        dict(corpus=np.array([3], np.int32), thr=None, kw=dict(sentence_len=1000)),
        dict(corpus=inputs.zipf_ids(3000, V, 1.0, 37), thr=None,
             kw=dict(sentence_len=1000, pos_begin=1000, pos_end=1000)),
        dict(corpus=inputs.zipf_ids(3000, V, 1.0, 38), thr=np.zeros(V, np.uint32),
             kw=dict(sentence_len=100)),
        dict(corpus=inputs.zipf_ids(3000, V, 1.0, 39), thr=None, kw=dict(sentence_len=1)),
    ]
    for case in cases:
        c = case["corpus"]
        gi, go, stats, _ = gpu_epoch(c, table, case["thr"], M_in, M_out, window=3, K=2,
                                     algorithm=algorithm, **case["kw"])
        begin = case["kw"].get("pos_begin", 0)
        end = case["kw"].get("pos_end", len(c))
        assert stats[0] == 0 and stats[1] == 0 and stats[2] == end - begin
        if case["thr"] is not None:
            # threshold 0 keeps only draws equal to 0: almost surely none
            mb = oracle.minibatches(oracle.Sampling(c, table, case["thr"], window=3, K=2,
                                                    **case["kw"]))
            assert len(mb["targets"]) == 0
        assert np.array_equal(gi.view(np.uint32), M_in.view(np.uint32))
        assert np.array_equal(go.view(np.uint32), M_out.view(np.uint32))


def test_out_of_range_corpus_ids_are_skipped_not_applied():
    """Ids outside [0, V) in the corpus are dropped before windows are formed;
    -1 (a word removed from the vocabulary) is no error, the others are
    counted as rejected and reported once as W2V_EDEVICE_FLAG."""
    V, D = 300, 32
    corpus = inputs.zipf_ids(8000, V, 1.0, 40)
    bad = corpus.copy()
    bad[[10, 1500, 4321]] = [V, -1, V + 7]
    table, _ = oracle.build_tables(inputs.word_counts(corpus, V), 0.75, 0.0, 10**6,
                                   want_thresh=False)
    M_in = inputs.init_matrix(V, D, "uniform", 41)
    M_out = inputs.init_matrix(V, D, "normal", 42, scale=0.05)
    gi, go, stats, _ = gpu_epoch(bad, table, None, M_in, M_out, window=4, K=3,
                                 sentence_len=1000, seed=43, max_inflight=1)
    assert stats[3] == 2 and stats[2] == len(bad)
    expect_device_flag()
    assert np.isfinite(gi).all() and np.isfinite(go).all()
    assert not np.array_equal(gi.view(np.uint32), M_in.view(np.uint32))


def test_dropped_words_equal_subsampled_positions():
    """A corpus position holding -1 (a word the vocabulary dropped) leaves
    its sentence before windows form, exactly as a position that subsampling
    rejects: the serialised epoch equals the oracle's epoch over the same
    corpus with an extra word V in those positions whose keep threshold is 0
    (kept only on a draw of exactly 0, which none of these positions has).
    The word V has count 0, so it owns no slot of the negative table and the
    table is the same. Nothing is reported as an error."""
    V, D, L = 300, 32, 100
    kw = dict(window=3, K=3, sentence_len=L, seed=48)
    corpus = inputs.zipf_ids(6000, V, 1.0, 44)
    drop = np.zeros(len(corpus), bool)
    drop[np.random.default_rng(45).integers(0, len(corpus), 400)] = True
    assert all(oracle.draw_u32(kw["seed"], int(p), 0, 0) != 0 for p in np.nonzero(drop)[0])
    table, _ = oracle.build_tables(inputs.word_counts(corpus, V), 0.75, 0.0, 10**6,
                                   want_thresh=False)
    M_in = inputs.init_matrix(V, D, "uniform", 46)
    M_out = inputs.init_matrix(V, D, "normal", 47, scale=0.05)
    gi, go, stats, _ = gpu_epoch(np.where(drop, -1, corpus).astype(np.int32), table, None,
                                 M_in, M_out, max_inflight=1, **kw)
    assert stats[3] == 0
    w2v.device_status()
    o_corpus = np.where(drop, V, corpus).astype(np.int32)
    thr = np.full(V + 1, 0xFFFFFFFF, np.uint32)
    thr[V] = 0
    o_in = np.vstack([M_in, np.zeros((1, D), np.float32)])
    o_out = np.vstack([M_out, np.zeros((1, D), np.float32)])
    n, _ = oracle.train_epoch(oracle.Sampling(o_corpus, table, thr, **kw), o_in, o_out)
    assert stats[0] == n
    assert rel_row_error(gi, o_in[:V]) < 2e-4
    assert rel_row_error(go, o_out[:V]) < 2e-4
    assert not o_in[V].any() and not o_out[V].any()


def test_dropped_minibatch_is_reported_to_a_caller_without_stats():
    """A caller that passes no stats learns of a skipped minibatch: the next
    call on the device returns W2V_EDEVICE_FLAG and launches nothing, the
    call after it runs."""
    import torch
    V, D = 200, 32
    corpus = inputs.zipf_ids(3000, V, 1.0, 49)
    corpus[1234] = V + 3
    table, _ = oracle.build_tables(inputs.word_counts(np.clip(corpus, 0, V - 1), V), 0.75,
                                   0.0, 10**5, want_thresh=False)
    gi = to_dev(inputs.init_matrix(V, D, "uniform", 50))
    go = torch.zeros_like(gi)
    c, tb = to_dev(corpus), to_dev(table)
    w2v.train_epoch(c, gi, go, tb, None, window=3, K=2)
    torch.cuda.synchronize()
    before = gi.clone()
    with pytest.raises(w2v.W2VError) as err:
        w2v.train_epoch(c, gi, go, tb, None, window=3, K=2)
    assert err.value.code == w2v.EDEVICE_FLAG
    torch.cuda.synchronize()
    assert torch.equal(gi, before)              # the reporting call launched nothing
    good = to_dev(np.clip(corpus, 0, V - 1).astype(np.int32))
    w2v.train_epoch(good, gi, go, tb, None, window=3, K=2)
    w2v.device_status()



def test_default_concurrency_caps():
    """Reading R24: the default launch is the wavefronts the GPU holds, capped
    by the vocabulary (V / (4 G (2 window + K + 1))) and by K (131072 /
    (K + 1), the bound under which the 10^6-word epoch stayed finite at
    K = 64)."""
    held = w2v.default_inflight(300, 5, 5, V=10**9)   # no vocabulary or K cap binds
    assert held >= 2048
    assert w2v.default_inflight(300, 5, 5, V=10**6) == held
    # K = 64: 131072 / 65 = 2016, below what the GPU holds for either D
    assert w2v.default_inflight(100, 5, 64, V=10**6) == 131072 // 65
    assert w2v.default_inflight(300, 5, 64, V=10**6) == 131072 // 65
    assert w2v.default_inflight(64, 5, 5, V=1000) == 1000 // (4 * 16)
    assert w2v.default_inflight(64, 5, 5, V=1000, group=4) == max(1, 1000 // (4 * 4 * 16))
