"""The throughput workload's shapes and launch configuration (V = 1e6
Zipf(1.07) words, D = 300 in rows padded to 320 floats, K = 5, window 5,
t = 1e-4, a 1e8-slot table, the conflict model's atomic rows and split head)
on prefixes of the benchmark's corpus that the oracle can follow:

* serialised, the first 1e6 tokens: elementwise against the oracle on every
  row the minibatches touch, every other row bitwise unchanged;
* as the benchmark launches it (every sentence of 1e7 tokens, 2048 in
  flight): minibatch and input-word counts equal the oracle's exactly, rows
  no minibatch touches stay bitwise unchanged, the matrices stay finite and
  the training loss falls along the epoch.
"""
import numpy as np
import pytest

import oracle
from gpu_util import to_dev
from paper_1611_06172_amd import inputs, w2v
from test_gpu_train_epoch import rel_row_error

pytestmark = pytest.mark.gpu

V, D = 1_000_000, 300


def workload(T):
    # the first T tokens of the throughput benchmark's own corpus (same
    # generator and seed), with tables from the law's expected counts
    corpus = inputs.zipf_corpus_hashed(T, V, 1.07, 6).numpy()
    counts = np.rint(inputs.zipf_pmf(V, 1.07) * 1e9).astype(np.int64)
    table, thr = oracle.build_tables(counts, 0.75, 1e-4, 10**8)
    M_in = inputs.init_matrix(V, D, "uniform", 2)
    inflight = w2v.default_inflight(D, 5, 5, V=V)
    hot = w2v.hot_rows(counts, inflight=inflight, tol=0.5)
    split = w2v.hot_rows(counts, inflight=inflight, tol=128.0)
    return corpus, table, thr, M_in, hot, split


def touched_rows(mb):
    t_in = np.unique(mb["ctx"][mb["ctx"] >= 0])
    t_out = np.unique(np.concatenate([mb["targets"], mb["negs"].ravel()]))
    return t_in, t_out


def run_gpu(corpus, table, thr, M_in, hot, split, **kw):
    import torch
    gi = w2v.alloc_matrix(V, D, "cuda", torch.from_numpy(M_in))
    go = w2v.alloc_matrix(V, D, "cuda")
    stats = torch.zeros(5, dtype=torch.int64, device="cuda")
    lb = torch.zeros((10, 2), dtype=torch.float64, device="cuda")
    w2v.train_epoch(to_dev(corpus), gi, go, to_dev(table),
                    torch.from_numpy(thr.view(np.int32)).cuda(), window=5, K=5,
                    seed=1234, stats=stats, loss_buckets=lb, hot_rows=hot,
                    split_rows=split, **kw)
    torch.cuda.synchronize()
    assert gi.stride(0) == 320
    return gi.cpu().numpy(), go.cpu().numpy(), stats.cpu().numpy(), lb.cpu().numpy()


def test_serialised_prefix_at_throughput_shapes():
    corpus, table, thr, M_in, hot, split = workload(1_000_000)
    assert hot > 1000 and split >= 1
    s = oracle.Sampling(corpus, table, thr, window=5, K=5, seed=1234)
    o_in, o_out = M_in.copy(), np.zeros_like(M_in)
    n, _ = oracle.train_epoch(s, o_in, o_out)
    gi, go, stats, _ = run_gpu(corpus, table, thr, M_in, hot, split, max_inflight=1)
    assert stats[0] == n and stats[2] == len(corpus) and stats[3] == 0
    t_in, t_out = touched_rows(oracle.minibatches(s))
    assert rel_row_error(gi[t_in], o_in[t_in]) < 2e-4
    assert rel_row_error(go[t_out], o_out[t_out]) < 2e-4
    rest_in = np.setdiff1d(np.arange(V), t_in)
    rest_out = np.setdiff1d(np.arange(V), t_out)
    assert np.array_equal(gi[rest_in].view(np.uint32), M_in[rest_in].view(np.uint32))
    assert not go[rest_out].any()


def test_bench_launch_configuration_on_a_prefix():
    corpus, table, thr, M_in, hot, split = workload(10_000_000)
    s = oracle.Sampling(corpus, table, thr, window=5, K=5, seed=1234)
    mb = oracle.minibatches(s)
    # the benchmark's concurrency (a default launch over only 1e4 sentences
    # would run fewer at once, to keep 8 rounds)
    gi, go, stats, lb = run_gpu(corpus, table, thr, M_in, hot, split,
                                max_inflight=w2v.default_inflight(D, 5, 5, V=V))
    assert stats[0] == len(mb["targets"])
    assert stats[1] == (mb["ctx"] >= 0).sum()
    assert stats[2] == len(corpus) and stats[3] == 0
    t_in, t_out = touched_rows(mb)
    rest_in = np.setdiff1d(np.arange(V), t_in)
    rest_out = np.setdiff1d(np.arange(V), t_out)
    assert np.array_equal(gi[rest_in].view(np.uint32), M_in[rest_in].view(np.uint32))
    assert not go[rest_out].any()
    assert np.isfinite(gi).all() and np.isfinite(go).all()
    loss = lb[:, 0] / lb[:, 1]
    assert loss[-1] < 0.9 * loss[0]
