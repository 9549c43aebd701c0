"""The throughput workload's shapes and launch configuration (V = 1e6
Zipf(1.07) words, D = 300 in rows padded to 320 floats, K = 5, window 5,
t = 1e-4, a 1e8-slot table, the conflict model's atomic rows and split head)
on prefixes of the benchmark's corpus that the oracle can follow:

* serialised, the first 1e6 tokens: elementwise against the oracle on every
  row the minibatches touch, every other row bitwise unchanged;
* as the benchmark launches it (every sentence of 1e7 tokens, 2048 in
  flight): minibatch and input-word counts equal the oracle's exactly, rows
  no minibatch touches stay bitwise unchanged, the matrices stay finite and
  the training loss falls along the epoch;
* the whole 1e9-token corpus as the benchmark trains it, and every cell of
  the shape sweep (D in {100, 300, 600} x K in {5, 15, 64}) on its 1e8-token
  corpus: per tenth of the corpus the epoch's input-word count equals the
  sampling export's over the same tenth (and the totals), the export equals
  the oracle bit for bit on sampled ranges at the start, middle and end, the
  matrices stay finite and the loss falls.
"""
import numpy as np
import pytest

import oracle
from gpu_util import assert_same_minibatches, gpu_minibatches, to_dev
from paper_1611_06172_amd import configs, inputs, w2v
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


def full_run(T, D_, K_, algorithm="hogbatch", group=1):
    """Trains the first T tokens of the throughput corpus for one epoch as
    bench.py does (tables from their counts, the default concurrency, the
    conflict model's atomic rows at tol 0.5 and at most two split rows),
    then checks it against the sampling export per tenth of the range and
    the export against the oracle on three sampled ranges."""
    import torch
    cfg = configs.LargeVocab()
    seed = cfg.sampling_seed
    print(f"[full] drawing {T} tokens, D {D_}, K {K_}", flush=True)
    corpus = inputs.zipf_corpus_hashed(T, V, cfg.zipf_s, cfg.corpus_seed, "cuda")
    counts = torch.bincount(corpus, minlength=V).cpu().numpy().astype(np.int64)
    table, thr = oracle.build_tables(counts, 0.75, cfg.sample, cfg.table_size)
    g_table, g_thr = w2v.build_tables(counts, 0.75, cfg.sample, cfg.table_size)
    assert np.array_equal(table, g_table) and np.array_equal(thr, g_thr)
    table_d, thr_d = to_dev(table), torch.from_numpy(thr.view(np.int32)).cuda()
    inflight = w2v.default_inflight(D_, cfg.window, K_, V=V, group=group)
    hot = w2v.hot_rows(counts, inflight=inflight, K=K_, tol=0.5)
    split = min(2, w2v.hot_rows(counts, inflight=inflight, K=K_, tol=128.0))
    if algorithm == "pairwise":
        split = 0   # partial rows serve the HogBatch kernels only
    gi = w2v.alloc_matrix(V, D_, "cuda",
                          torch.from_numpy(inputs.init_matrix(V, D_, "uniform", cfg.init_seed)))
    go = w2v.alloc_matrix(V, D_, "cuda")
    stats = torch.zeros(5, dtype=torch.int64, device="cuda")
    lb = torch.zeros((10, 2), dtype=torch.float64, device="cuda")
    print(f"[full] epoch: inflight {inflight}, hot {hot}, split {split}", flush=True)
    w2v.train_epoch(corpus, gi, go, table_d, thr_d, window=cfg.window, K=K_,
                    seed=seed, stats=stats, loss_buckets=lb, max_inflight=inflight,
                    hot_rows=hot, split_rows=split, algorithm=algorithm, group=group)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(gi).all()) and bool(torch.isfinite(go).all())
    del gi, go
    st, lbh = stats.cpu().numpy(), lb.cpu().numpy()
    kw = dict(V=V, window=cfg.window, K=K_, seed=seed)
    step = T // 10
    n_tot = in_tot = 0
    for b in range(10):
        mb = w2v.debug_minibatches(corpus, table_d, thr_d, pos_begin=b * step,
                                   pos_end=(b + 1) * step, **kw)
        keep = mb["targets"] >= 0
        n_b = int(keep.sum())
        in_b = int(((mb["ctx"] >= 0).sum(1) * keep).sum())
        del mb
        assert lbh[b, 1] == in_b, (b, lbh[b, 1], in_b)
        n_tot += n_b
        in_tot += in_b
    print(f"[full] {n_tot} minibatches, {in_tot} input words", flush=True)
    assert st[0] == n_tot and st[1] == in_tot and st[2] == T and st[3] == 0
    corpus_h = corpus.cpu().numpy()
    for b0 in (0, T // 2, T - 200_000):
        o = oracle.minibatches(oracle.Sampling(corpus_h, table, thr, window=cfg.window,
                                               K=K_, seed=seed, pos_begin=b0,
                                               pos_end=b0 + 200_000))
        g = gpu_minibatches(w2v.debug_minibatches(corpus, table_d, thr_d, pos_begin=b0,
                                                  pos_end=b0 + 200_000, **kw), b0)
        assert_same_minibatches(g, o)
    # the loss per input word starts at (K + 1) ln 2 (M_out = 0) and every
    # later tenth is below the first one
    loss = lbh[:, 0] / lbh[:, 1]
    print(f"[full] loss per tenth {np.round(loss, 4).tolist()}", flush=True)
    assert loss[0] < (K_ + 1) * np.log(2.0)
    assert loss[1:].max() < loss[0]
    return loss


def test_whole_corpus_in_the_bench_launch():
    """The 1e9-token throughput workload (D = 300, K = 5), as bench.py runs it."""
    cfg = configs.LargeVocab()
    loss = full_run(cfg.T, cfg.D, cfg.K)
    assert loss[-1] < loss[0] - 0.1


@pytest.mark.parametrize("D_,K_", [(d, k) for d in configs.Sweep().dims
                                   for k in configs.Sweep().negatives])
def test_sweep_cell_at_full_size(D_, K_):
    """Each cell of the shape sweep on its 1e8-token corpus, as bench.py
    --tokens 1e8 --dim D --negative K runs it."""
    full_run(configs.Sweep().T, D_, K_)


@pytest.mark.parametrize("algorithm,group", [("hogbatch", 2), ("hogbatch", 4),
                                             ("pairwise", 1), ("hogbatch_immediate", 1)])
def test_other_variants_at_full_size(algorithm, group):
    """The variants bench.py measures beside the headline (negatives shared by
    2 and 4 targets, Algorithm 1, write-back at the end of each minibatch) on
    the 1e8-token corpus in their bench launch: the same targets and input
    words as the sampling export, finite matrices, a falling loss."""
    full_run(configs.Sweep().T, configs.LargeVocab().D, configs.LargeVocab().K,
             algorithm=algorithm, group=group)
