"""The memory-ceiling measurement kernel behind `bench.py --workload
row-rmw`: it must perform exactly the accesses it claims. With one
wavefront and distinct rows within each step, every row ends up increased
by the number of times it was drawn; with many wavefronts and every row
updated atomically, too (repeats within a step included)."""
import ctypes
import os

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def lib():
    L = ctypes.CDLL(os.path.join(ROOT, "paper_1611_06172_amd", "libw2v_measure.so"))
    L.w2v_measure_row_rmw.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                      ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                      ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                      ctypes.c_void_p]
    return L


@pytest.mark.parametrize("grid,atomic_rows", [(1, 0), (1, 3), (256, 12)])
def test_row_updates_are_exact(grid, atomic_rows):
    import torch
    V, D, ld, rows, n_steps = 500, 300, 320, 12, 3000
    rng = np.random.default_rng(grid + atomic_rows)
    if atomic_rows == rows:
        ids = rng.integers(0, V, n_steps * rows)       # repeats within a step
    else:
        ids = np.concatenate([rng.permutation(V)[:rows] for _ in range(n_steps)])
    M = torch.zeros((V, ld), dtype=torch.float32, device="cuda")
    t = torch.from_numpy(ids.astype(np.int32)).cuda()
    rc = lib().w2v_measure_row_rmw(M.data_ptr(), V, D, ld, t.data_ptr(), n_steps, rows,
                                   atomic_rows, grid, torch.cuda.current_stream().cuda_stream)
    assert rc == 0
    torch.cuda.synchronize()
    got = M.cpu().numpy()
    want = np.bincount(ids, minlength=V).astype(np.float32)
    assert np.array_equal(got[:, :D], np.repeat(want[:, None], D, 1))
    assert not got[:, D:].any()


def test_invalid_arguments_are_refused():
    import torch
    M = torch.zeros((10, 64), device="cuda")
    t = torch.zeros(24, dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    L = lib()
    assert L.w2v_measure_row_rmw(M.data_ptr(), 10, 64, 64, t.data_ptr(), 2, 17, 0, 1, s) == -1
    assert L.w2v_measure_row_rmw(M.data_ptr(), 10, 64, 32, t.data_ptr(), 2, 12, 0, 1, s) == -1
    assert L.w2v_measure_row_rmw(M.data_ptr(), 10, 64, 64, t.data_ptr(), 2, 12, 13, 1, s) == -1
