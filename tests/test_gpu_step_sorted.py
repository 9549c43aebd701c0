"""w2v_step_batch_sorted: the snapshot batch with each row's updates summed
in a fixed order (staging rows, stable radix sort by row id, chunked fp64
sums added in chunk order).

Against the oracle with the bar of the atomic snapshot batch (see
test_gpu_step_batch.py); two runs from the same inputs give the same bits;
the atomic batch agrees to fp64 rounding of the sums. Cases: the
kernel-test configuration at full size, the eight shapes of the atomic
batch's tests (D = 1 .. 640, padded rows, N up to 32, K up to 64, K = 0),
absent inputs and masked negatives, a few rows shared by every minibatch
(runs that cross thousands of chunks), and out-of-range ids.
"""
import numpy as np
import pytest

import oracle
from paper_1611_06172_amd import inputs, w2v
from gpu_util import scaled_error, to_dev, expect_device_flag
from test_gpu_step_batch import TOL, check, mats

pytestmark = pytest.mark.gpu


def run(t, c, n, M_in, M_out, alpha, D=None, sorted=True):
    import torch
    gi, go = to_dev(M_in), to_dev(M_out)
    w2v.step_batch(to_dev(t), to_dev(c), to_dev(n), gi, go, alpha, D=D, sorted=sorted)
    torch.cuda.synchronize()
    return gi.cpu().numpy(), go.cpu().numpy()


def test_kernel_test_config_full_size_and_reproducible():
    t, c, n = inputs.kernel_batch(65536, 10, 5, 100_000, 1.0, 3)
    M_in, M_out = mats(100_000, 300, 4)
    print("[sorted] kernel-test configuration", flush=True)
    gi, go, stats = check(t, c, n, M_in, M_out, 0.025, sorted=True)
    assert stats[0] == 65536 and stats[1] == 65536 * 10
    ri, ro = run(t, c, n, M_in, M_out, 0.025)
    assert np.array_equal(ri.view(np.uint32), gi.view(np.uint32))
    assert np.array_equal(ro.view(np.uint32), go.view(np.uint32))
    ai, ao = run(t, c, n, M_in, M_out, 0.025, sorted=False)
    for g, a in ((gi, ai), (go, ao)):
        d = np.abs(g.astype(np.float64) - a)
        assert d.max() <= 1e-6 * np.abs(a).max()
        assert (d > 0).mean() < 1e-3   # last-bit differences only, and rarely


@pytest.mark.parametrize("V,D,ld,B,N,K", [
    (500, 100, 100, 3000, 10, 5),
    (700, 64, 64, 2000, 10, 5),
    (300, 1, 1, 500, 4, 3),
    (400, 300, 320, 1500, 10, 5),
    (200, 640, 640, 300, 10, 5),
    (900, 200, 200, 1000, 16, 25),
    (600, 100, 100, 800, 32, 64),
    (50, 96, 96, 400, 6, 0),
    (6, 300, 320, 2000, 10, 5),    # six rows: every run crosses many chunks
])
def test_shapes(V, D, ld, B, N, K):
    print(f"[sorted] V={V} D={D} ld={ld} B={B} N={N} K={K}", flush=True)
    t, c, n = inputs.kernel_batch(B, N, K, V, 1.0, V + D)
    M_in, M_out = mats(V, D, 7, ld=ld)
    check(t, c, n, M_in, M_out, 0.03, D=D, sorted=True)


def test_absent_inputs_masks_and_per_minibatch_alpha():
    V, D, B = 120, 72, 900
    t, c, n = inputs.kernel_batch(B, 8, 5, V, 1.0, 21)
    rng = np.random.default_rng(0)
    c[rng.random(c.shape) < 0.3] = -1
    c[:40] = -1
    n[::7, 2] = t[::7]
    alpha = rng.uniform(0.001, 0.05, B).astype(np.float32)
    check(t, c, n, *mats(V, D, 9), alpha, sorted=True)


@pytest.mark.parametrize("shared", [(3, 1, 2, 2, 5, 0), (40, 41, 42, 42, 45, 8)])
def test_rows_shared_by_every_minibatch(shared):
    """Every minibatch has the same target and negatives: their runs span
    every chunk of the output sort, and the head rows of the inputs most
    (the head ids of a Zipf law, then ids from the middle of the range)."""
    V, D, B = 64, 300, 4096
    t = np.full(B, shared[0], np.int32)
    c = inputs.zipf_ids((B, 10), V, 0.5, 5)
    n = np.tile(np.array([shared[1:]], np.int32), (B, 1))
    check(t, c, n, *mats(V, D, 11), 0.001, sorted=True)


def test_bad_ids_are_skipped():
    import torch
    V, D, B = 100, 64, 64
    t, c, n = inputs.kernel_batch(B, 5, 3, V, 1.0, 31)
    t[3] = V
    c[10, 2] = -7
    n[20, 0] = 1 << 30
    Mi, Mo = mats(V, D, 13)
    keep = np.ones(B, bool)
    keep[[3, 10, 20]] = False
    Mi_o, Mo_o, S_in, S_out = oracle.step_batch(t[keep], c[keep], n[keep], Mi, Mo, 0.02)
    gi, go = to_dev(Mi), to_dev(Mo)
    stats = torch.zeros(5, dtype=torch.int64, device="cuda")
    w2v.step_batch(to_dev(t), to_dev(c), to_dev(n), gi, go, 0.02, stats=stats, sorted=True)
    torch.cuda.synchronize()
    assert stats[3].item() == 3 and stats[0].item() == B - 3
    expect_device_flag()
    assert scaled_error(gi.cpu().numpy(), Mi_o, S_in) <= TOL
    assert scaled_error(go.cpu().numpy(), Mo_o, S_out) <= TOL


def test_empty_batch_and_validation():
    import torch
    M = torch.zeros((10, 8), device="cuda")
    e = torch.empty((0,), dtype=torch.int32, device="cuda")
    w2v.step_batch(e, e.view(0, 4), e.view(0, 2), M, M.clone(), sorted=True)
    with pytest.raises(w2v.W2VError):
        ws = torch.empty(16, dtype=torch.uint8, device="cuda")
        t = torch.zeros(2, dtype=torch.int32, device="cuda")
        w2v.step_batch(t, t.view(2, 1), t.view(2, 1), M, M.clone(), workspace=ws,
                       sorted=True)
