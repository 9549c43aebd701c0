"""Pending input-row updates (LDS slots of the HogBatch epoch kernel).

A cold input row's updates collect in a slot while its word is in the
window and reach M_in in one atomic add when the slot is released. With one
sentence in flight that changes only the order of the fp32 additions
(m + (g1 + g2) instead of (m + g1) + g2), so the pending and immediate
kernels agree to rounding, and both against the oracle's sequential epoch.
Covered here: slot counts, agreement across shapes and update tiers
(including minibatches with more distinct inputs than slots, several output
blocks and ragged sentences), that nothing stays pending after a call
(sentence-aligned chunks equal one call bit for bit, untouched rows keep
their bits), and that the grouped kernel ignores the choice.
"""
import numpy as np
import pytest

import oracle
from paper_1611_06172_amd import inputs, w2v
from gpu_util import to_dev, thresh_dev

pytestmark = pytest.mark.gpu


def run(corpus, table, thr, M_in, M_out, algorithm, **kw):
    import torch
    gi, go = to_dev(M_in), to_dev(M_out)
    stats = torch.zeros(5, dtype=torch.int64, device="cuda")
    w2v.train_epoch(to_dev(corpus), gi, go, to_dev(table), thresh_dev(thr),
                    stats=stats, algorithm=algorithm, **kw)
    torch.cuda.synchronize()
    return gi.cpu().numpy(), go.cpu().numpy(), stats.cpu().numpy()


def rel_row_error(g, o):
    """max over elements of |g - o| / (max |o| in the row + 1e-3 * max |o|)."""
    d = np.abs(g.astype(np.float64) - o)
    scale = np.abs(o).max(axis=1, keepdims=True) + 1e-3 * np.abs(o).max()
    return float((d / scale).max())


@pytest.mark.parametrize("D,window,K", [(300, 5, 5), (64, 5, 5), (600, 5, 5),
                                        (200, 8, 25), (72, 16, 1), (128, 16, 64)])
def test_slot_count(D, window, K):
    n = w2v.pending_slots(D, window, K)
    print(f"[pending] D={D} window={window} K={K}: {n} slots", flush=True)
    assert 2 <= n <= 16


CASES = [
    (1000, 64, 5, 5, 0.0, 1000, 0, 0),       # every row cold
    (600, 100, 2, 5, 1e-3, 257, 0, 0),       # window 2, ragged sentences
    (300, 200, 8, 3, 0.0, 1000, 0, 0),       # 16 inputs: more than the slots
    (200, 72, 16, 1, 1e-2, 1024, 0, 0),      # 32 inputs, blocks of 2
    (3000, 300, 5, 25, 1e-3, 1000, 0, 0),    # several output blocks
    (1000, 300, 5, 5, 0.0, 1000, 40, 0),     # atomic head rows
    (1000, 64, 5, 5, 0.0, 1000, 37, 3),      # split head rows
    (800, 600, 5, 5, 1e-3, 1000, 30, 0),     # 10 columns per lane
    (700, 100, 5, 15, 0.0, 1000, 0, 2),      # 2 columns, several output blocks
]


@pytest.mark.parametrize("V,D,window,K,sub,L,hot,split", CASES)
def test_pending_matches_immediate_and_oracle_serialised(V, D, window, K, sub, L, hot, split):
    corpus = inputs.zipf_ids(30_000, V, 1.0, V + window + K)
    table, thr = oracle.build_tables(inputs.word_counts(corpus, V), 0.75, sub, 10**6)
    if sub == 0.0:
        thr = None
    M_in = inputs.init_matrix(V, D, "uniform", 3)
    M_out = inputs.init_matrix(V, D, "normal", 4, scale=0.05)
    kw = dict(window=window, K=K, sentence_len=L, seed=9)
    print(f"[pending] V={V} D={D} window={window} K={K} hot={hot} split={split}",
          flush=True)
    pi, po, ps = run(corpus, table, thr, M_in, M_out, "hogbatch", max_inflight=1,
                     hot_rows=hot, split_rows=split, **kw)
    ii, io, is_ = run(corpus, table, thr, M_in, M_out, "hogbatch_immediate",
                      max_inflight=1, hot_rows=hot, split_rows=split, **kw)
    assert np.array_equal(ps, is_)
    assert rel_row_error(pi, ii.astype(np.float64)) < 2e-5
    assert rel_row_error(po, io.astype(np.float64)) < 2e-5
    o_in, o_out = M_in.copy(), M_out.copy()
    oracle.train_epoch(oracle.Sampling(corpus, table, thr, **kw), o_in, o_out)
    assert rel_row_error(pi, o_in) < 2e-4
    assert rel_row_error(po, o_out) < 2e-4


def test_nothing_pending_after_a_call():
    """Two sentence-aligned calls equal one call bit for bit (every slot is
    flushed at the end of its sentence), and words absent from the corpus
    keep their rows' bits."""
    import torch
    V, D = 500, 64
    corpus = inputs.zipf_ids(30_000, 250, 1.0, 12)          # ids < 250 only
    table, _ = oracle.build_tables(inputs.word_counts(corpus, V), 0.75, 0.0, 10**6,
                                   want_thresh=False)
    M_in = inputs.init_matrix(V, D, "uniform", 3)
    M_out = inputs.init_matrix(V, D, "normal", 4, scale=0.05)
    kw = dict(window=5, K=5, sentence_len=1000, seed=2, max_inflight=1, hot_rows=0)
    a_in, a_out, _ = run(corpus, table, None, M_in, M_out, "hogbatch", **kw)
    gi, go = to_dev(M_in), to_dev(M_out)
    c, tb = to_dev(corpus), to_dev(table)
    for b, e in ((0, 12_000), (12_000, 30_000)):
        w2v.train_epoch(c, gi, go, tb, None, pos_begin=b, pos_end=e, **kw)
    torch.cuda.synchronize()
    assert np.array_equal(gi.cpu().numpy().view(np.uint32), a_in.view(np.uint32))
    assert np.array_equal(go.cpu().numpy().view(np.uint32), a_out.view(np.uint32))
    assert np.array_equal(a_in[250:].view(np.uint32), M_in[250:].view(np.uint32))
    assert not np.array_equal(a_in[:250], M_in[:250])


def test_grouped_ignores_the_choice():
    V, D = 1000, 64
    corpus = inputs.zipf_ids(20_000, V, 1.0, 21)
    table, _ = oracle.build_tables(inputs.word_counts(corpus, V), 0.75, 0.0, 10**6,
                                   want_thresh=False)
    M_in = inputs.init_matrix(V, D, "uniform", 3)
    M_out = inputs.init_matrix(V, D, "normal", 4, scale=0.05)
    kw = dict(window=5, K=5, sentence_len=1000, seed=9, max_inflight=1, group=4,
              hot_rows=0)
    pi, po, _ = run(corpus, table, None, M_in, M_out, "hogbatch", **kw)
    ii, io, _ = run(corpus, table, None, M_in, M_out, "hogbatch_immediate", **kw)
    assert np.array_equal(pi.view(np.uint32), ii.view(np.uint32))
    assert np.array_equal(po.view(np.uint32), io.view(np.uint32))
