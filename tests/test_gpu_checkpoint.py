"""Resume and failure detection on the GPU path: an epoch run in checkpointed
ranges, cut short and resumed, equals the uncut serialised epoch bit for bit
(matrices and loss buckets); a checkpoint of another configuration is
refused; a NaN planted in a matrix row is flagged by w2v_check_loss through
the loss buckets of the minibatches that read it."""
import numpy as np
import pytest

import oracle
from gpu_util import to_dev
from paper_1611_06172_amd import checkpoint, inputs, w2v

pytestmark = pytest.mark.gpu

V, D, T = 1000, 64, 60_000


def setup():
    import torch
    corpus = inputs.zipf_ids(T, V, 1.0, 1).astype(np.int32)
    table, thr = oracle.build_tables(inputs.word_counts(corpus, V), 0.75, 1e-3, 10**6)
    M0 = inputs.init_matrix(V, D, "uniform", 2)
    return (to_dev(corpus), to_dev(table), torch.from_numpy(thr.view(np.int32)).cuda(), M0)


def test_resumed_epoch_is_bitwise_the_uncut_epoch(tmp_path):
    import torch
    corpus, table, thr, M0 = setup()
    kw = dict(window=5, K=5, epoch=1, n_epochs=2, seed=5, max_inflight=1)
    ref_in, ref_out = to_dev(M0), torch.zeros((V, D), device="cuda")
    ref_loss = torch.zeros((6, 2), dtype=torch.float64, device="cuda")
    w2v.train_epoch(corpus, ref_in, ref_out, table, thr, loss_buckets=ref_loss, **kw)
    torch.cuda.synchronize()

    path = str(tmp_path / "ck")
    gi, go = to_dev(M0), torch.zeros((V, D), device="cuda")
    lb = torch.zeros((6, 2), dtype=torch.float64, device="cuda")
    rec = checkpoint.train_epoch_resumable(path, corpus, gi, go, table, thr,
                                           chunk_sentences=7, loss_buckets=lb,
                                           max_chunks=4, **kw)
    assert rec["next_pos"] == 4 * 7 * 1000
    # a fresh process would start from new tensors: the checkpoint restores them
    gi2, go2 = to_dev(M0), torch.zeros((V, D), device="cuda")
    lb2 = torch.zeros((6, 2), dtype=torch.float64, device="cuda")
    rec = checkpoint.train_epoch_resumable(path, corpus, gi2, go2, table, thr,
                                           chunk_sentences=7, loss_buckets=lb2, **kw)
    assert rec["next_pos"] == T
    torch.cuda.synchronize()
    assert torch.equal(gi2.view(torch.int32), ref_in.view(torch.int32))
    assert torch.equal(go2.view(torch.int32), ref_out.view(torch.int32))
    assert torch.equal(lb2[:, 1], ref_loss[:, 1])
    assert torch.allclose(lb2[:, 0], ref_loss[:, 0], rtol=1e-12, atol=0)
    # the epoch is done: a further call changes nothing
    again = checkpoint.train_epoch_resumable(path, corpus, gi2, go2, table, thr,
                                             chunk_sentences=7, loss_buckets=lb2, **kw)
    assert again["generation"] == rec["generation"]
    # another seed is another configuration
    with pytest.raises(ValueError):
        checkpoint.train_epoch_resumable(path, corpus, gi2, go2, table, thr,
                                         chunk_sentences=7, loss_buckets=lb2,
                                         **dict(kw, seed=6))


def test_nan_in_a_row_is_flagged_through_the_loss():
    import torch
    corpus, table, thr, M0 = setup()
    lb = torch.zeros((4, 2), dtype=torch.float64, device="cuda")
    gi, go = to_dev(M0), torch.zeros((V, D), device="cuda")
    w2v.train_epoch(corpus, gi, go, table, thr, window=5, K=5, seed=3, loss_buckets=lb)
    w2v.check_loss(lb)                      # a clean run passes
    M = M0.copy()
    M[0, 3] = np.nan                        # the most frequent word's input row
    gi, go = to_dev(M), torch.zeros((V, D), device="cuda")
    lb.zero_()
    w2v.train_epoch(corpus, gi, go, table, thr, window=5, K=5, seed=3, loss_buckets=lb)
    with pytest.raises(w2v.W2VError) as e:
        w2v.check_loss(lb)
    assert e.value.code == w2v.ENONFINITE and "loss bucket 0" in str(e.value)
