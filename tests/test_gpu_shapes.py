"""The shape sweep's shapes (D in {100, 300, 600} x K in {5, 15, 64},
window 5): serialised epochs of both algorithms against the oracle, on a
Zipf(1.07) stream over a vocabulary small enough for the oracle. These
cover one and several output blocks (K + 1 = 6, 16, 65 against blocks of 6),
two and ten columns per lane (D = 100 -> 2, 600 -> 10), and padded rows."""
import numpy as np
import pytest

import oracle
from gpu_util import to_dev
from paper_1611_06172_amd import inputs, w2v
from test_gpu_train_epoch import rel_row_error

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("algorithm", ["hogbatch", "pairwise"])
@pytest.mark.parametrize("D", [100, 300, 600])
@pytest.mark.parametrize("K", [5, 15, 64])
def test_sweep_shape_serialised(D, K, algorithm):
    import torch
    V = 3000
    T = 6000 if (D * K >= 300 * 15) else 12_000
    corpus = inputs.zipf_ids(T, V, 1.07, 7)
    table, thr = oracle.build_tables(inputs.word_counts(corpus, V), 0.75, 1e-4, 10**7)
    M_in = inputs.init_matrix(V, D, "uniform", 8)
    M_out = inputs.init_matrix(V, D, "normal", 9, scale=0.02)
    kw = dict(window=5, K=K, sentence_len=1000, seed=10)
    o_in, o_out = M_in.copy(), M_out.copy()
    run = oracle.pairwise_train_epoch if algorithm == "pairwise" else oracle.train_epoch
    n, ob = run(oracle.Sampling(corpus, table, thr, **kw), o_in, o_out, n_buckets=2)
    gi = w2v.alloc_matrix(V, D, "cuda", torch.from_numpy(M_in))
    go = w2v.alloc_matrix(V, D, "cuda", torch.from_numpy(M_out))
    stats = torch.zeros(5, dtype=torch.int64, device="cuda")
    lb = torch.zeros((2, 2), dtype=torch.float64, device="cuda")
    w2v.train_epoch(to_dev(corpus), gi, go, to_dev(table),
                    torch.from_numpy(thr.view(np.int32)).cuda(), loss_buckets=lb,
                    stats=stats, max_inflight=1, hot_rows=100, algorithm=algorithm, **kw)
    torch.cuda.synchronize()
    assert int(stats[0]) == n
    assert rel_row_error(gi.cpu().numpy(), o_in) < 2e-4
    assert rel_row_error(go.cpu().numpy(), o_out) < 2e-4
    gb = lb.cpu().numpy()
    np.testing.assert_array_equal(gb[:, 1], ob[:, 1])
    np.testing.assert_allclose(gb[:, 0], ob[:, 0], rtol=1e-5)
