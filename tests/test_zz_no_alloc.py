"""w2v_train_epoch_noalloc, the entry point for callers that cannot allocate
(its split rows' partial rows live in the library's static device scratch
array), against w2v_train_epoch with a caller-owned workspace, through the
C ABI: two calls in a row, the second with a smaller input (fewer words,
shorter rows, fewer split rows), so that the scratch contents the first
call leaves behind must not leak into the second. Serialised epochs run the
same kernels in the same order, so the matrices must agree bit for bit; a
concurrent epoch is compared against the oracle's sequential one within
the statistical bar. An oversized request is rejected before any launch."""
import numpy as np
import pytest

import oracle
from gpu_util import to_dev
from paper_1611_06172_amd import inputs, w2v

pytestmark = pytest.mark.gpu


def case(V, D, T, seed):
    import torch
    corpus = inputs.zipf_ids(T, V, 1.0, seed)
    table, thr = oracle.build_tables(inputs.word_counts(corpus, V), 0.75, 1e-3, 10**6)
    M_in = inputs.init_matrix(V, D, "uniform", seed + 1)
    M_out = inputs.init_matrix(V, D, "normal", seed + 2, scale=0.02)
    dev = dict(corpus=to_dev(corpus), table=to_dev(table),
               thr=torch.from_numpy(thr.view(np.int32)).cuda())
    return corpus, table, thr, M_in, M_out, dev


def padded(M):
    import torch
    return w2v.alloc_matrix(M.shape[0], M.shape[1], "cuda", torch.from_numpy(M))


@pytest.mark.parametrize("inflight", [1, 0])
def test_noalloc_matches_the_workspace_entry_point_on_two_calls(inflight):
    import torch
    w2v.init()
    for V, D, T, split, seed in ((3000, 300, 40_000, 60, 61), (800, 100, 15_000, 9, 71)):
        corpus, table, thr, M_in, M_out, dev = case(V, D, T, seed)
        kw = dict(window=5, K=5, sentence_len=1000, seed=seed, max_inflight=inflight,
                  hot_rows=40, split_rows=split)
        a_in, a_out = padded(M_in), padded(M_out)
        b_in, b_out = padded(M_in), padded(M_out)
        ws_bytes = w2v.train_epoch_workspace_bytes(split, a_in.stride(0))
        assert 0 < ws_bytes <= w2v.NOALLOC_SCRATCH_BYTES
        sa = torch.zeros(5, dtype=torch.int64, device="cuda")
        sb = torch.zeros(5, dtype=torch.int64, device="cuda")
        w2v.train_epoch(dev["corpus"], a_in, a_out, dev["table"], dev["thr"], stats=sa,
                        **kw)
        w2v.train_epoch_noalloc(dev["corpus"], b_in, b_out, dev["table"], dev["thr"],
                                stats=sb, **kw)
        torch.cuda.synchronize()
        print(f"[noalloc] V={V} D={D} split={split} inflight={inflight}", flush=True)
        assert torch.equal(sa, sb)
        if inflight == 1:
            assert torch.equal(a_in.view(torch.int32), b_in.view(torch.int32))
            assert torch.equal(a_out.view(torch.int32), b_out.view(torch.int32))
        else:
            # concurrent: Hogwild order differs run to run; both against the
            # oracle's sequential epoch
            o_in, o_out = M_in.copy(), M_out.copy()
            oracle.train_epoch(oracle.Sampling(corpus, table, thr, window=5, K=5,
                                               sentence_len=1000, seed=seed), o_in, o_out)
            hb_t, hb_c, _ = inputs.kernel_batch(1000, 6, 5, V, 1.0, 99)
            hb_n = table[np.random.default_rng(98).integers(0, len(table), (1000, 5))]
            from test_gpu_train_epoch import eval_loss
            lo = eval_loss(o_in, o_out, hb_t, hb_c, hb_n)
            for gi, go in ((a_in, a_out), (b_in, b_out)):
                lg = eval_loss(gi.cpu().numpy(), go.cpu().numpy(), hb_t, hb_c, hb_n)
                assert abs(lg - lo) <= 0.02 * lo, (lg, lo)
    w2v.device_status()


def test_noalloc_rejects_split_rows_beyond_the_scratch():
    import torch
    w2v.init()
    V, D = 1000, 300
    corpus, table, thr, M_in, M_out, dev = case(V, D, 5000, 81)
    g_in, g_out = padded(M_in), padded(M_out)
    ld = g_in.stride(0)
    too_many = w2v.NOALLOC_SCRATCH_BYTES // (2 * 8 * ld * 4) + 1
    assert w2v.train_epoch_workspace_bytes(too_many, ld) > w2v.NOALLOC_SCRATCH_BYTES
    with pytest.raises(w2v.W2VError) as err:
        w2v.train_epoch_noalloc(dev["corpus"], g_in, g_out, dev["table"], dev["thr"],
                                split_rows=too_many)
    assert err.value.code == w2v.EINVAL and "scratch" in str(err.value)
    torch.cuda.synchronize()
    assert np.array_equal(g_in.cpu().numpy().view(np.uint32), M_in.view(np.uint32))
