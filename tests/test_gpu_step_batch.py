"""w2v_step_batch against the oracle's snapshot batch.

Bar: for every element |gpu - oracle| <= 1e-5 * S, where the oracle computes
in fp64 and rounds once, and S = |M0| + the sum, over every occurrence of the
row in the batch, of the absolute products forming that occurrence's update
(sum_k |E_ik| |O_kj| for M_in, sum_i |E_ik| |A_ij| for M_out) -- the scale of
the rounding error of evaluating those sums of products in fp32. The GPU sums
the occurrences in fp64 and rounds once, like the oracle, so accumulation
order does not enter. Rows the batch does not touch are bitwise unchanged,
and so are padding columns D..ld-1.
"""
import numpy as np
import pytest

import oracle
from paper_1611_06172_amd import inputs, w2v
from gpu_util import scaled_error, to_dev, expect_device_flag

pytestmark = pytest.mark.gpu
TOL = 1e-5


def check(targets, contexts, negatives, M_in, M_out, alpha, D=None, expect_skip=0,
          sorted=False):
    import torch
    V, ld = M_in.shape
    D = ld if D is None else D
    Mi_o, Mo_o, S_in, S_out = oracle.step_batch(targets, contexts, negatives,
                                                M_in, M_out, alpha, D=D)
    gi, go = to_dev(M_in), to_dev(M_out)
    a = to_dev(alpha) if np.ndim(alpha) else alpha
    stats = torch.zeros(5, dtype=torch.int64, device="cuda")
    w2v.step_batch(to_dev(targets), to_dev(contexts), to_dev(negatives), gi, go,
                   a, D=D, stats=stats, sorted=sorted)
    torch.cuda.synchronize()
    gi, go = gi.cpu().numpy(), go.cpu().numpy()
    for name, g, o, S, M0 in (("M_in", gi, Mi_o, S_in, M_in),
                              ("M_out", go, Mo_o, S_out, M_out)):
        err = scaled_error(g[:, :D], o[:, :D], S)
        d = np.abs(g[:, :D].astype(np.float64) - o[:, :D])
        rel = d / np.maximum(np.abs(o[:, :D]), 1e-30)
        print(f"{name}: max scaled error {err:.3e}, max abs {d.max():.3e}, "
              f"elements with plain relative error > 1e-5: {(rel > 1e-5).mean():.2e}")
        assert err <= TOL
        untouched = np.all(o == M0, axis=1)
        assert np.array_equal(g[untouched].view(np.uint32), M0[untouched].view(np.uint32))
        if ld > D:
            assert np.array_equal(g[:, D:].view(np.uint32), M0[:, D:].view(np.uint32))
    assert stats[3].item() == expect_skip
    return gi, go, stats.cpu().numpy()


def mats(V, D, seed, ld=None, kind="normal"):
    return (inputs.init_matrix(V, D, kind, seed, ld=ld),
            inputs.init_matrix(V, D, kind, seed + 100, ld=ld))


def test_kernel_test_config_full_size():
    """B = 65,536 minibatches, N = 10, K = 5, Zipf(1.0) ids over V = 100,000,
    D = 300, M ~ N(0, 0.1^2), alpha = 0.025."""
    t, c, n = inputs.kernel_batch(65536, 10, 5, 100_000, 1.0, 3)
    M_in, M_out = mats(100_000, 300, 4)
    _, _, stats = check(t, c, n, M_in, M_out, 0.025)
    assert stats[0] == 65536 and stats[1] == 65536 * 10


@pytest.mark.parametrize("V,D,ld,B,N,K", [
    (500, 100, 100, 3000, 10, 5),    # two column blocks, ragged second
    (700, 64, 64, 2000, 10, 5),      # one full column block
    (300, 1, 1, 500, 4, 3),          # D = 1
    (400, 300, 320, 1500, 10, 5),    # padded rows
    (200, 640, 640, 300, 10, 5),     # largest D
    (900, 200, 200, 1000, 16, 25),   # window-8 shape, several output blocks
    (600, 100, 100, 800, 32, 64),    # largest N and K
    (50, 96, 96, 400, 6, 0),         # no negatives
])
def test_shapes(V, D, ld, B, N, K):
    t, c, n = inputs.kernel_batch(B, N, K, V, 1.0, V + D)
    M_in, M_out = mats(V, D, 7, ld=ld)
    check(t, c, n, M_in, M_out, 0.03, D=D)


def test_absent_inputs_masks_and_per_minibatch_alpha():
    V, D, B = 120, 72, 900
    t, c, n = inputs.kernel_batch(B, 8, 5, V, 1.0, 21)
    rng = np.random.default_rng(0)
    c[rng.random(c.shape) < 0.3] = -1        # absent input words
    c[:40] = -1                               # empty minibatches are no-ops
    n[::7, 2] = t[::7]                        # negatives equal to the target
    alpha = rng.uniform(0.001, 0.05, B).astype(np.float32)
    check(t, c, n, *mats(V, D, 9), alpha)


def test_hot_rows():
    """Every minibatch shares the same target and negatives: maximal atomic
    contention on a handful of rows."""
    V, D, B = 64, 300, 4096
    t = np.full(B, 3, np.int32)
    c = inputs.zipf_ids((B, 10), V, 0.5, 5)
    n = np.tile(np.array([[1, 2, 2, 5, 0]], np.int32), (B, 1))
    check(t, c, n, *mats(V, D, 11), 0.001)


def test_bad_ids_are_skipped():
    V, D, B = 100, 64, 64
    t, c, n = inputs.kernel_batch(B, 5, 3, V, 1.0, 31)
    t[3] = V
    c[10, 2] = -7
    n[20, 0] = 1 << 30
    Mi, Mo = mats(V, D, 13)
    keep = np.ones(B, bool)
    keep[[3, 10, 20]] = False
    Mi_o, Mo_o, S_in, S_out = oracle.step_batch(t[keep], c[keep], n[keep], Mi, Mo, 0.02)
    import torch
    gi, go = to_dev(Mi), to_dev(Mo)
    stats = torch.zeros(5, dtype=torch.int64, device="cuda")
    w2v.step_batch(to_dev(t), to_dev(c), to_dev(n), gi, go, 0.02, stats=stats)
    torch.cuda.synchronize()
    assert stats[3].item() == 3 and stats[0].item() == B - 3
    expect_device_flag()
    assert scaled_error(gi.cpu().numpy(), Mi_o, S_in) <= TOL
    assert scaled_error(go.cpu().numpy(), Mo_o, S_out) <= TOL


def test_empty_batch_and_validation():
    import torch
    M = torch.zeros((10, 8), device="cuda")
    e = torch.empty((0,), dtype=torch.int32, device="cuda")
    w2v.step_batch(e, e.view(0, 4), e.view(0, 2), M, M.clone())
    with pytest.raises(w2v.W2VError):
        big = torch.zeros((2, 33), dtype=torch.int32, device="cuda")
        w2v.step_batch(big[:, 0].contiguous(), big, big[:, :2].contiguous(), M, M.clone())
    with pytest.raises(w2v.W2VError):
        ws = torch.empty(16, dtype=torch.uint8, device="cuda")
        t = torch.zeros(2, dtype=torch.int32, device="cuda")
        w2v.step_batch(t, t.view(2, 1), t.view(2, 1), M, M.clone(), workspace=ws)


def test_strided_views_are_rejected():
    """The kernels read contexts, negatives and loss buckets as packed
    arrays; a strided view would be read at the wrong places, so the
    binding refuses it (the row-padded matrices, whose stride is passed as
    ld, are the only strided arguments)."""
    import torch
    V, D = 50, 16
    M_in = torch.zeros((V, D), device="cuda")
    M_out = torch.zeros((V, D), device="cuda")
    t = torch.zeros(8, dtype=torch.int32, device="cuda")
    wide = torch.zeros((8, 12), dtype=torch.int32, device="cuda")
    negs = torch.zeros((8, 3), dtype=torch.int32, device="cuda")
    with pytest.raises(ValueError):
        w2v.step_batch(t, wide[:, :10], negs, M_in, M_out)
    with pytest.raises(ValueError):
        w2v.step_batch(t, wide[:, :4].contiguous(), wide[:, ::4], M_in, M_out)
    c = torch.zeros(3000, dtype=torch.int32, device="cuda")
    tb = torch.zeros(10, dtype=torch.int32, device="cuda")
    lb = torch.zeros((4, 3), dtype=torch.float64, device="cuda")[:, :2]
    with pytest.raises(ValueError):
        w2v.train_epoch(c, M_in, M_out, tb, loss_buckets=lb)
    # a padded matrix view is accepted
    P = w2v.alloc_matrix(V, D, "cuda")
    assert P.stride(0) == 32
    w2v.step_batch(t, wide[:, :4].contiguous(), negs, P, w2v.alloc_matrix(V, D, "cuda"))
