"""Checkpoint files (paper_1611_06172_amd/checkpoint.py) on the host, and
resume exactness shown with the oracle: an epoch cut at a sentence boundary,
saved, loaded and continued equals the uncut epoch bit for bit (every draw
depends on (seed, epoch, raw position) only)."""
import json
import os

import numpy as np
import pytest

import oracle
from paper_1611_06172_amd import checkpoint, inputs


def test_round_trip_generations_and_hash(tmp_path):
    p = str(tmp_path / "ck")
    a = np.arange(12, dtype=np.float32).reshape(3, 4)
    b = -a
    loss = np.array([[1.5, 2.0], [3.0, 4.0]])
    r0 = checkpoint.save(p, a, b, dict(seed=1, epoch=0, n_epochs=2, next_pos=1000,
                                       config_hash="h0"), loss_buckets=loss)
    assert r0["generation"] == 0
    r1 = checkpoint.save(p, a + 1, b, dict(seed=1, epoch=0, n_epochs=2, next_pos=2000,
                                           config_hash="h0"))
    assert r1["generation"] == 1 and "loss" not in r1["files"]
    # the older generation is gone, the new one complete
    names = sorted(os.listdir(p))
    assert names == sorted(["state.json", "M_in.1.npy", "M_out.1.npy"])
    rec, arr = checkpoint.load(p, expect_hash="h0")
    assert rec["next_pos"] == 2000
    assert np.array_equal(arr["M_in"], a + 1) and np.array_equal(arr["M_out"], b)
    with pytest.raises(ValueError):
        checkpoint.load(p, expect_hash="other")
    assert checkpoint.load(str(tmp_path / "none")) == (None, None)


def test_interrupted_save_keeps_the_last_complete_checkpoint(tmp_path):
    """A save cut short after writing its arrays but before replacing
    state.json leaves the previous record, which names complete arrays."""
    p = str(tmp_path / "ck")
    a = np.ones((2, 3), np.float32)
    checkpoint.save(p, a, a, dict(epoch=0, next_pos=10, config_hash="h"))
    # what a killed save of generation 1 leaves behind
    np.save(os.path.join(p, "M_in.1.npy"), a * 7)
    with open(os.path.join(p, "state.json.tmp"), "w") as f:
        f.write("{truncated")
    rec, arr = checkpoint.load(p, expect_hash="h")
    assert rec["generation"] == 0 and rec["next_pos"] == 10
    assert np.array_equal(arr["M_in"], a)


def test_config_hash_depends_on_config_and_arrays():
    t = np.arange(10, dtype=np.int32)
    h = checkpoint.config_hash({"K": 5, "window": 5}, t, None)
    assert h == checkpoint.config_hash({"window": 5, "K": 5}, t.copy(), None)
    assert h != checkpoint.config_hash({"K": 6, "window": 5}, t, None)
    assert h != checkpoint.config_hash({"K": 5, "window": 5}, t[::-1].copy(), None)
    assert h != checkpoint.config_hash({"K": 5, "window": 5}, t, t)
    c = np.arange(5_000_000, dtype=np.int32)
    f = checkpoint.corpus_fingerprint(c)
    c2 = c.copy()
    c2[-1] += 1
    assert f != checkpoint.corpus_fingerprint(c2)


def test_oracle_epoch_resumed_from_a_checkpoint_is_bitwise_the_uncut_epoch(tmp_path):
    V, D, T, L = 1000, 16, 30_000, 1000
    corpus = inputs.zipf_ids(T, V, 1.0, 1).astype(np.int32)
    counts = inputs.word_counts(corpus, V)
    table, thr = oracle.build_tables(counts, 0.75, 1e-3, 10**6)
    M0 = inputs.init_matrix(V, D, "uniform", 2)

    def samp(b, e):
        return oracle.Sampling(corpus=corpus, neg_table=table, keep_thresh=thr,
                               window=5, K=5, epoch=1, n_epochs=3, seed=9,
                               pos_begin=b, pos_end=e)

    full_in, full_out = M0.copy(), np.zeros_like(M0)
    _, full_loss = oracle.train_epoch(samp(0, T), full_in, full_out, n_buckets=4)

    mid = 13 * L
    part_in, part_out = M0.copy(), np.zeros_like(M0)
    _, loss_a = oracle.train_epoch(samp(0, mid), part_in, part_out, n_buckets=4)
    p = str(tmp_path / "ck")
    checkpoint.save(p, part_in, part_out,
                    dict(seed=9, epoch=1, n_epochs=3, next_pos=mid, config_hash="x"),
                    loss_buckets=loss_a)
    del part_in, part_out
    rec, arr = checkpoint.load(p, expect_hash="x")
    res_in, res_out = arr["M_in"].copy(), arr["M_out"].copy()
    _, loss_b = oracle.train_epoch(samp(rec["next_pos"], T), res_in, res_out, n_buckets=4)
    assert np.array_equal(res_in.view(np.uint32), full_in.view(np.uint32))
    assert np.array_equal(res_out.view(np.uint32), full_out.view(np.uint32))
    # buckets hold disjoint positions, so the two ranges' sums add up
    assert np.allclose(arr["loss"] + loss_b, full_loss, rtol=1e-12, atol=0)
    assert json.load(open(os.path.join(p, "state.json")))["next_pos"] == mid
