"""The first 1e8 tokens of the throughput benchmark's corpus
(tests/largevocab.py) trained as the benchmark launches it (V = 1e6,
D = 300 in rows padded to 320 floats, K = 5, window 5, t = 1e-4, 2048
sentences in flight, the conflict model's atomic rows at tol 0.5, at most
two split rows, the pending input-row slots) against the oracle's
sequential epoch over the same tokens: same minibatches and input counts per
bucket, the training loss per input word in each of ten buckets of raw
position and the held-out loss of the trained model within 2%. The oracle's
numbers come from tests/golden/make_largevocab_trajectory.py. The kernel that
writes every update back at the end of its minibatch (the paper's
write-back) runs the same comparison."""
import json
import os

import numpy as np
import pytest

import largevocab as lv
from paper_1611_06172_amd import inputs, w2v

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "largevocab_oracle.json")


def test_hashed_corpus_is_the_same_on_the_gpu():
    """The benchmark draws its corpus on the GPU, the stored oracle numbers
    use the same generator on the host: the ids agree."""
    import torch
    for begin in (0, 123_456_789):
        g = inputs.zipf_corpus_hashed(1 << 20, lv.V, 1.07, lv.CORPUS_SEED, "cuda", begin=begin)
        h = inputs.zipf_corpus_hashed(1 << 20, lv.V, 1.07, lv.CORPUS_SEED, "cpu", begin=begin)
        assert torch.equal(g.cpu(), h)


@pytest.mark.parametrize("algorithm", ["hogbatch", "hogbatch_immediate"])
def test_bench_launch_trajectory_matches_the_oracle(algorithm):
    import torch
    with open(GOLDEN) as f:
        golden = json.load(f)
    assert golden.get("complete"), "golden incomplete: rerun make_largevocab_trajectory.py"
    dev = torch.device("cuda")
    corpus = lv.corpus(dev)
    counts = torch.bincount(corpus, minlength=lv.V).cpu().numpy().astype(np.int64)
    table_h, thr_h = w2v.build_tables(counts, 0.75, lv.SAMPLE, 10**8)
    inflight = w2v.default_inflight(lv.D, lv.WINDOW, lv.K, V=lv.V)
    hot = w2v.hot_rows(counts, sample_t=lv.SAMPLE, inflight=inflight, tol=0.5)
    split = min(2, w2v.hot_rows(counts, sample_t=lv.SAMPLE, inflight=inflight, tol=128.0))
    M_in = w2v.alloc_matrix(lv.V, lv.D, dev, torch.from_numpy(lv.init_in()))
    M_out = w2v.alloc_matrix(lv.V, lv.D, dev)
    stats = torch.zeros(5, dtype=torch.int64, device=dev)
    lb = torch.zeros((lv.N_BUCKETS, 2), dtype=torch.float64, device=dev)
    print(f"[largevocab] {algorithm}: inflight {inflight}, hot {hot}, split {split}",
          flush=True)
    w2v.train_epoch(corpus, M_in, M_out, torch.from_numpy(table_h).to(dev),
                    torch.from_numpy(thr_h.view(np.int32)).to(dev), window=lv.WINDOW,
                    K=lv.K, seed=lv.SEED, stats=stats, loss_buckets=lb, hot_rows=hot,
                    split_rows=split, algorithm=algorithm)
    torch.cuda.synchronize()
    st, gb = stats.cpu().numpy(), lb.cpu().numpy()
    ob = np.array(golden["buckets"])
    assert st[0] == golden["minibatches"] and st[3] == 0
    np.testing.assert_array_equal(gb[:, 1], ob[:, 1])
    traj_o, traj_g = ob[:, 0] / ob[:, 1], gb[:, 0] / gb[:, 1]
    print(f"[largevocab] {algorithm}: buckets "
          f"{np.round(100 * (traj_g / traj_o - 1), 3).tolist()} %", flush=True)
    assert np.all(np.abs(traj_g - traj_o) <= 0.02 * traj_o), (traj_g, traj_o)
    held = lv.heldout_loss(M_in.cpu().numpy(), M_out.cpu().numpy(), *lv.heldout_ids(table_h))
    h = golden["heldout_after_range"][-1]
    print(f"[largevocab] {algorithm}: held-out {held:.5f} oracle {h:.5f}", flush=True)
    assert held < 0.9 * golden["heldout_loss_initial"]
    assert abs(held - h) <= 0.02 * h, (held, h)
