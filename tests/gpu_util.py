"""Helpers shared by the GPU parity tests (no arithmetic of the method)."""
import numpy as np


def to_dev(a, dtype=None):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def thresh_dev(thr):
    """uint32 thresholds as an int32 device tensor with the same bits."""
    import torch
    if thr is None:
        return None
    return torch.from_numpy(np.ascontiguousarray(thr).view(np.int32)).cuda()


def gpu_minibatches(out, pos_begin=0):
    """Compacts the per-position GPU export into the oracle's list layout."""
    t = out["targets"].cpu().numpy()
    idx = np.nonzero(t >= 0)[0]
    return dict(targets=t[idx], ctx=out["ctx"].cpu().numpy()[idx],
                negs=out["negs"].cpu().numpy()[idx],
                mask=out["mask"].cpu().numpy()[idx],
                alpha=out["alpha"].cpu().numpy()[idx],
                pos=(idx + pos_begin).astype(np.int64))


def assert_same_minibatches(g, o):
    assert g["targets"].shape == o["targets"].shape, (g["targets"].shape, o["targets"].shape)
    for key in ("pos", "targets", "ctx", "negs", "mask"):
        assert np.array_equal(g[key], o[key]), key
    assert np.array_equal(g["alpha"].view(np.uint32), o["alpha"].view(np.uint32))


def scaled_error(g, o, S):
    """max |g - o| / S over elements (S = |M0| + sum |update summands|)."""
    d = np.abs(g.astype(np.float64) - o.astype(np.float64))
    return float(np.max(d / np.maximum(S, 1e-300)))


def expect_device_flag():
    """Asserts that the library reports skipped work once (W2V_EDEVICE_FLAG
    from w2v_device_status, which waits for the stream) and that the report
    cleared the device's error word."""
    import pytest

    from paper_1611_06172_amd import w2v
    with pytest.raises(w2v.W2VError) as err:
        w2v.device_status()
    assert err.value.code == w2v.EDEVICE_FLAG
    w2v.device_status()
