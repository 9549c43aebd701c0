"""HogBatch with negatives shared by groups of G consecutive targets
(group = 2, 4, 8) against the oracle's grouped epoch.

* Serialised: elementwise, counts exact, loss buckets; shapes with one and
  several output blocks, subsampling, padded rows, the three update tiers.
* Hogwild: per-epoch training-loss trajectory and held-out loss within 2%.
"""
import numpy as np
import pytest

import oracle
from gpu_util import thresh_dev, to_dev
from paper_1611_06172_amd import inputs, w2v
from test_gpu_train_epoch import eval_loss, gpu_epoch, heldout_batch, rel_row_error, tiny_config

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("G,V,D,window,K,sub,L,hot,split,padded", [
    (2, 1000, 64, 5, 5, 0.0, 1000, None, 0, False),
    (4, 1000, 64, 5, 5, 0.0, 1000, 40, 3, False),
    (4, 2000, 300, 5, 5, 1e-3, 1000, 37, 1, True),
    (8, 600, 100, 3, 15, 0.0, 257, 0, 0, False),
    (8, 300, 72, 2, 0, 1e-2, 50, None, 0, False),
])
def test_serialised_grouped_matches_oracle(G, V, D, window, K, sub, L, hot, split, padded):
    import torch
    corpus = inputs.zipf_ids(25_000, V, 1.0, V + G)
    table, thr = oracle.build_tables(inputs.word_counts(corpus, V), 0.75, sub, 10**6)
    if sub == 0.0:
        thr = None
    M_in = inputs.init_matrix(V, D, "uniform", 51)
    M_out = inputs.init_matrix(V, D, "normal", 52, scale=0.05)
    kw = dict(window=window, K=K, sentence_len=L, seed=53)
    o_in, o_out = M_in.copy(), M_out.copy()
    n, ob = oracle.grouped_train_epoch(oracle.Sampling(corpus, table, thr, **kw), G,
                                       o_in, o_out, n_buckets=3)
    if padded:
        gi = w2v.alloc_matrix(V, D, "cuda", torch.from_numpy(M_in))
        go = w2v.alloc_matrix(V, D, "cuda", torch.from_numpy(M_out))
    else:
        gi, go = to_dev(M_in), to_dev(M_out)
    stats = torch.zeros(5, dtype=torch.int64, device="cuda")
    lb = torch.zeros((3, 2), dtype=torch.float64, device="cuda")
    w2v.train_epoch(to_dev(corpus), gi, go, to_dev(table), thresh_dev(thr), loss_buckets=lb,
                    stats=stats, max_inflight=1, hot_rows=hot, split_rows=split, group=G,
                    **kw)
    torch.cuda.synchronize()
    mb = oracle.minibatches(oracle.Sampling(corpus, table, thr, **kw))
    st = stats.cpu().numpy()
    assert st[0] == n and st[1] == (mb["ctx"] >= 0).sum() and st[3] == 0
    assert rel_row_error(gi.cpu().numpy(), o_in) < 2e-4
    assert rel_row_error(go.cpu().numpy(), o_out) < 2e-4
    gb = lb.cpu().numpy()
    np.testing.assert_array_equal(gb[:, 1], ob[:, 1])
    np.testing.assert_allclose(gb[:, 0], ob[:, 0], rtol=1e-5)


@pytest.mark.parametrize("G", [2, 4])
def test_grouped_tiny_configuration_default_launch_trajectory(G):
    """The tiny configuration (200,000 tokens over 1,000 words, D = 64,
    window 5, K = 5, one epoch) with groups of G targets, launched by
    default: the library caps the concurrent sentences at V / (4 G (2 window
    + K + 1)) (7 for G = 2, 3 for G = 4), because a group's step reads rows
    G targets old and so multiplies the staleness of concurrency. The
    training loss per input word in ten buckets of raw position and the
    held-out loss within 2% of the sequential grouped oracle's."""
    V, D = 1000, 64
    corpus, table, M_in, M_out = tiny_config(V=V, D=D)
    assert w2v.default_inflight(D, 5, 5, V=V, group=G) == V // (4 * G * 16)
    kw = dict(window=5, K=5, sentence_len=1000, seed=55, alpha0=0.025, n_epochs=1)
    o_in, o_out = M_in.copy(), M_out.copy()
    _, ob = oracle.grouped_train_epoch(oracle.Sampling(corpus, table, None, **kw), G,
                                       o_in, o_out, n_buckets=10)
    gi, go, _, gb = gpu_epoch(corpus, table, None, M_in, M_out, n_buckets=10, group=G,
                              **kw)
    np.testing.assert_array_equal(gb[:, 1], ob[:, 1])
    traj_o, traj_g = ob[:, 0] / ob[:, 1], gb[:, 0] / gb[:, 1]
    print(f"[grouped default] G={G}: buckets "
          f"{np.round(100 * (traj_g / traj_o - 1), 2).tolist()} %", flush=True)
    assert np.all(np.abs(traj_g - traj_o) <= 0.02 * traj_o), (traj_g, traj_o)
    hb = heldout_batch(V, table)
    lo, lg = eval_loss(o_in, o_out, *hb), eval_loss(gi, go, *hb)
    assert abs(lg - lo) <= 0.02 * lo, (lg, lo)


def test_stress_grouped_small_vocabulary_many_in_flight():
    """Stress test, outside the statistical bar: G = 4 over 1,000 words with
    64 sentences in flight (21 times the default concurrency for this
    vocabulary). Observed: epoch-0 training loss 17% above the sequential
    grouped epoch. Checked here: the run stays finite and learns."""
    V, D = 1000, 64
    corpus, table, M_in, M_out = tiny_config(V=V, D=D)
    kw = dict(window=5, K=5, sentence_len=1000, seed=55, alpha0=0.025, n_epochs=1)
    gi, go, _, gb = gpu_epoch(corpus, table, None, M_in, M_out, n_buckets=10, group=4,
                              max_inflight=64, **kw)
    assert np.isfinite(gi).all() and np.isfinite(go).all()
    traj = gb[:, 0] / gb[:, 1]
    assert traj[-1] < 0.9 * traj[0]
    hb = heldout_batch(V, table)
    assert eval_loss(gi, go, *hb) < 0.95 * eval_loss(M_in, M_out, *hb)


@pytest.mark.parametrize("G", [2, 4])
def test_hogwild_grouped_near_sequential(G):
    """64 sentences in flight over 20,000 words, three epochs (observed
    within 0.5%)."""
    import torch
    V = 20_000
    corpus, table, M_in, M_out = tiny_config(T=400_000, V=V)
    E = 3
    kw = dict(window=5, K=5, sentence_len=1000, seed=54, alpha0=0.025, n_epochs=E)
    o_in, o_out = M_in.copy(), M_out.copy()
    gi, go = to_dev(M_in), to_dev(M_out)
    c, tb = to_dev(corpus), to_dev(table)
    traj_o, traj_g = [], []
    for e in range(E):
        _, ob = oracle.grouped_train_epoch(oracle.Sampling(corpus, table, None, epoch=e, **kw),
                                           G, o_in, o_out, n_buckets=1)
        lb = torch.zeros((1, 2), dtype=torch.float64, device="cuda")
        w2v.train_epoch(c, gi, go, tb, None, epoch=e, loss_buckets=lb, max_inflight=64,
                        group=G, **kw)
        gb = lb.cpu().numpy()
        assert gb[0, 1] == ob[0, 1]
        traj_o.append(ob[0, 0] / ob[0, 1])
        traj_g.append(gb[0, 0] / gb[0, 1])
    traj_o, traj_g = np.array(traj_o), np.array(traj_g)
    assert traj_o[-1] < traj_o[0]
    assert np.all(np.abs(traj_g - traj_o) <= 0.02 * traj_o), (traj_g, traj_o)
    t, ctx, _ = inputs.kernel_batch(2000, 6, 5, V, 1.0, 99)
    negs = table[np.random.default_rng(98).integers(0, len(table), (2000, 5))]
    lo = eval_loss(o_in, o_out, t, ctx, negs)
    lg = eval_loss(gi.cpu().numpy(), go.cpu().numpy(), t, ctx, negs)
    assert abs(lg - lo) <= 0.02 * lo, (lg, lo)
