"""The Algorithm 1 epoch (algorithm="pairwise", the paper's per-pair Hogwild
baseline) against the oracle's sequential Algorithm 1.

* Serialised (max_inflight = 1): elementwise, fp32 versus fp64 rounding
  bound as for the HogBatch epoch; shapes cover one and several output
  blocks (K up to 64), K = 0, subsampling, window 8 and 16, ragged
  sentences, padded rows, and the atomic and plain update paths. Counts are
  exact.
* Hogwild: the per-epoch training-loss trajectory and the final held-out
  loss within 2% of the sequential oracle's.
"""
import numpy as np
import pytest

import oracle
from gpu_util import thresh_dev, to_dev
from paper_1611_06172_amd import inputs, w2v
from test_gpu_train_epoch import eval_loss, rel_row_error, tiny_config

pytestmark = pytest.mark.gpu


def gpu_pairwise(corpus, table, thr, M_in, M_out, n_buckets=0, ld=None, **kw):
    import torch
    if ld is None:
        gi, go = to_dev(M_in), to_dev(M_out)
    else:
        gi = w2v.alloc_matrix(*M_in.shape, "cuda", torch.from_numpy(M_in))
        go = w2v.alloc_matrix(*M_out.shape, "cuda", torch.from_numpy(M_out))
    stats = torch.zeros(5, dtype=torch.int64, device="cuda")
    lb = torch.zeros((n_buckets, 2), dtype=torch.float64, device="cuda") if n_buckets else None
    w2v.train_epoch(to_dev(corpus), gi, go, to_dev(table), thresh_dev(thr),
                    loss_buckets=lb, stats=stats, algorithm="pairwise", **kw)
    torch.cuda.synchronize()
    return (gi.cpu().numpy(), go.cpu().numpy(), stats.cpu().numpy(),
            None if lb is None else lb.cpu().numpy())


@pytest.mark.parametrize("V,D,window,K,sub,L,hot,padded", [
    (1000, 64, 5, 5, 0.0, 1000, None, False),   # tiny configuration, one block
    (2000, 300, 5, 5, 1e-3, 1000, 37, True),    # subsampling, mixed paths, ld 320
    (600, 100, 8, 25, 0.0, 257, 0, False),      # 4 blocks of outputs, plain stores
    (300, 72, 16, 64, 1e-2, 1024, None, False), # 9 blocks, window 16
    (500, 40, 3, 0, 0.0, 50, None, False),      # no negatives, short sentences
])
def test_serialised_pairwise_matches_oracle(V, D, window, K, sub, L, hot, padded):
    corpus = inputs.zipf_ids(25_000, V, 1.0, V + K)
    table, thr = oracle.build_tables(inputs.word_counts(corpus, V), 0.75, sub, 10**6)
    if sub == 0.0:
        thr = None
    M_in = inputs.init_matrix(V, D, "uniform", 21)
    M_out = inputs.init_matrix(V, D, "normal", 22, scale=0.05)
    kw = dict(window=window, K=K, sentence_len=L, seed=23)
    o_in, o_out = M_in.copy(), M_out.copy()
    n, ob = oracle.pairwise_train_epoch(oracle.Sampling(corpus, table, thr, **kw),
                                        o_in, o_out, n_buckets=3)
    gi, go, stats, gb = gpu_pairwise(corpus, table, thr, M_in, M_out, n_buckets=3,
                                     ld=320 if padded else None, max_inflight=1,
                                     hot_rows=hot, **kw)
    mb = oracle.minibatches(oracle.Sampling(corpus, table, thr, **kw))
    assert stats[0] == n and stats[1] == (mb["ctx"] >= 0).sum() and stats[3] == 0
    assert rel_row_error(gi, o_in) < 2e-4
    assert rel_row_error(go, o_out) < 2e-4
    np.testing.assert_array_equal(gb[:, 1], ob[:, 1])
    np.testing.assert_allclose(gb[:, 0], ob[:, 0], rtol=1e-5)


def test_pairwise_single_input_word_equals_hogbatch_on_gpu():
    """Two-token sentences and a one-word table: Algorithm 1 and HogBatch are
    the same computation, on the GPU as in the oracle."""
    import torch
    V, D = 50, 64
    corpus = inputs.zipf_ids(4000, V - 1, 1.0, 24)
    table = np.full(1000, V - 1, np.int32)
    M_in = inputs.init_matrix(V, D, "uniform", 25)
    M_out = inputs.init_matrix(V, D, "normal", 26, scale=0.2)
    kw = dict(window=3, K=1, sentence_len=2, seed=27, max_inflight=1)
    a_in, a_out, _, _ = gpu_pairwise(corpus, table, None, M_in, M_out, **kw)
    h_in, h_out = to_dev(M_in), to_dev(M_out)
    w2v.train_epoch(to_dev(corpus), h_in, h_out, to_dev(table), None, **kw)
    torch.cuda.synchronize()
    assert rel_row_error(a_in, h_in.cpu().numpy().astype(np.float64)) < 1e-5
    assert rel_row_error(a_out, h_out.cpu().numpy().astype(np.float64)) < 1e-5


def test_hogwild_pairwise_near_sequential():
    import torch
    corpus, table, M_in, M_out = tiny_config()
    E = 3
    kw = dict(window=5, K=5, sentence_len=1000, seed=28, alpha0=0.025, n_epochs=E)
    o_in, o_out = M_in.copy(), M_out.copy()
    gi, go = to_dev(M_in), to_dev(M_out)
    c, tb = to_dev(corpus), to_dev(table)
    traj_o, traj_g = [], []
    for e in range(E):
        _, ob = oracle.pairwise_train_epoch(
            oracle.Sampling(corpus, table, None, epoch=e, **kw), o_in, o_out, n_buckets=1)
        lb = torch.zeros((1, 2), dtype=torch.float64, device="cuda")
        w2v.train_epoch(c, gi, go, tb, None, epoch=e, loss_buckets=lb, max_inflight=64,
                        algorithm="pairwise", **kw)
        gb = lb.cpu().numpy()
        assert gb[0, 1] == ob[0, 1]
        traj_o.append(ob[0, 0] / ob[0, 1])
        traj_g.append(gb[0, 0] / gb[0, 1])
    traj_o, traj_g = np.array(traj_o), np.array(traj_g)
    assert traj_o[-1] < traj_o[0]
    assert np.all(np.abs(traj_g - traj_o) <= 0.02 * traj_o), (traj_g, traj_o)
    t, ctx, _ = inputs.kernel_batch(2000, 6, 5, 1000, 1.0, 99)
    negs = table[np.random.default_rng(98).integers(0, len(table), (2000, 5))]
    lo = eval_loss(o_in, o_out, t, ctx, negs)
    lg = eval_loss(gi.cpu().numpy(), go.cpu().numpy(), t, ctx, negs)
    assert abs(lg - lo) <= 0.02 * lo, (lg, lo)


def test_pairwise_rejects_split_rows():
    import torch
    c = torch.zeros(100, dtype=torch.int32, device="cuda")
    M = torch.zeros((10, 8), device="cuda")
    tb = torch.zeros(4, dtype=torch.int32, device="cuda")
    with pytest.raises(w2v.W2VError):
        w2v.train_epoch(c, M, M.clone(), tb, split_rows=1, algorithm="pairwise")
