"""Host-side checks of libw2v that need no GPU: the library loads, exports
every entry point include/w2v.h declares, builds the same tables as the oracle
bit for bit, and rejects invalid arguments before touching the device."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_1611_06172_amd import inputs, w2v

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    with open(os.path.join(ROOT, "include", "w2v.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(w2v_[a-z_0-9]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 7
    L = w2v.lib()
    for name in names:
        assert hasattr(L, name), name


def test_version():
    assert w2v.version() == 104


@pytest.mark.parametrize("seed,power,t,size", [
    (0, 0.75, 1e-4, 10**6), (1, 0.75, 0.0, 12345), (2, 1.0, 1e-2, 10**7),
    (3, 0.5, 1e-3, 2**31 + 11)])
def test_tables_equal_oracle(seed, power, t, size):
    rng = np.random.default_rng(seed)
    counts = rng.integers(0, 10**6, 3000).astype(np.int64)
    counts[::13] = 0
    big = size > 10**8
    ta, ka = w2v.build_tables(counts, power, t, size, want_table=not big)
    tb, kb = oracle.build_tables(counts, power, t, size, want_table=not big)
    if not big:
        assert np.array_equal(ta, tb)
    assert np.array_equal(ka, kb)


def test_tables_large_vocab_equal_oracle():
    V = 1_000_000
    counts = np.rint(inputs.zipf_pmf(V, 1.07) * 1e9).astype(np.int64)
    ta, ka = w2v.build_tables(counts, 0.75, 1e-4, 10**8)
    tb, kb = oracle.build_tables(counts, 0.75, 1e-4, 10**8)
    assert np.array_equal(ta, tb) and np.array_equal(ka, kb)


def test_table_arguments_rejected():
    with pytest.raises(w2v.W2VError):
        w2v.build_tables(np.array([-1, 3], np.int64))
    with pytest.raises(w2v.W2VError):
        w2v.build_tables(np.zeros(4, np.int64))
    with pytest.raises(w2v.W2VError):
        w2v.build_tables(np.ones(4, np.int64), table_size=2**32)
    assert "table_size" in w2v.lib().w2v_last_error().decode()


# Fake, never-dereferenced device addresses: validation must fail first.
FAKE = 0x1000


def train(**over):
    args = dict(corpus=FAKE, T=1000, pos_begin=0, pos_end=1000, L=100, M_in=FAKE,
                M_out=FAKE, V=10, D=8, ld=8, window=5, K=5, table=FAKE,
                table_size=100, thr=None, alpha0=0.025, minf=1e-4, epoch=0,
                n_epochs=1, seed=0, loss=None, n_b=0, stats=None, inflight=0,
                hot=0, split=0, ws=None, ws_bytes=0, algorithm=0, group=1, stream=None)
    args.update(over)
    return w2v.lib().w2v_train_epoch(*args.values())


@pytest.mark.parametrize("over,needle", [
    (dict(corpus=None), "corpus"), (dict(T=0), "T"), (dict(L=0), "sentence_len"),
    (dict(L=1025), "sentence_len"), (dict(pos_begin=50), "pos_begin"),
    (dict(pos_end=950), "pos_end"), (dict(pos_begin=200, pos_end=100), "pos_begin"),
    (dict(V=0), "V"), (dict(D=0), "D"), (dict(D=641, ld=641), "D"),
    (dict(ld=7), "ld"), (dict(window=0), "window"), (dict(window=17), "window"),
    (dict(K=-1), "K"), (dict(K=65), "K"), (dict(table_size=2**32), "table_size"),
    (dict(table=None), "neg_table"), (dict(epoch=1), "epoch"),
    (dict(n_epochs=0), "epoch"), (dict(M_in=None), "M_in"),
    (dict(loss=FAKE, n_b=0), "n_buckets"), (dict(inflight=-1), "max_inflight"),
    (dict(hot=-1), "hot_rows"), (dict(split=-1), "split_rows"),
    (dict(split=11), "split_rows"), (dict(split=2), "workspace"),
    (dict(split=2, ws=0x100000, ws_bytes=2 * 2 * 8 * 8 * 4 - 1), "workspace"),
    (dict(split=2, ws=0x100010, ws_bytes=1 << 20), "aligned"),
    (dict(algorithm=3), "algorithm"), (dict(algorithm=-1), "algorithm"),
    (dict(algorithm=1, split=1, ws=0x100000, ws_bytes=1 << 20), "pairwise"),
    (dict(group=3), "group"), (dict(group=0), "group"), (dict(group=16), "group"),
    (dict(group=2, algorithm=1), "group"), (dict(group=8, window=5), "group"),
    (dict(group=8, window=2, K=30), "group"), (dict(group=2, window=16, K=5), "group"),
])
def test_train_epoch_rejects(over, needle):
    assert train(**over) == w2v.EINVAL
    assert needle in w2v.lib().w2v_last_error().decode()


def step(**over):
    args = dict(B=4, N=10, K=5, t=FAKE, c=FAKE, n=FAKE, alpha=None, a_s=0.025,
                M_in=FAKE, M_out=FAKE, V=10, D=8, ld=8, ws=0x100000, ws_bytes=1 << 20,
                stats=None, stream=None)
    args.update(over)
    return w2v.lib().w2v_step_batch(*args.values())


@pytest.mark.parametrize("over,needle", [
    (dict(B=-1), "B"), (dict(N=33), "N"), (dict(K=65), "K"), (dict(t=None), "targets"),
    (dict(c=None), "contexts"), (dict(n=None), "negatives"), (dict(ws=None), "workspace"),
    (dict(ws_bytes=100), "workspace"), (dict(ws=0x100010), "aligned"),
    (dict(D=700, ld=700), "D"), (dict(ld=4), "ld"),
])
def test_step_batch_rejects(over, needle):
    assert step(**over) == w2v.EINVAL
    assert needle in w2v.lib().w2v_last_error().decode()


def test_workspace_size():
    assert w2v.step_batch_workspace_bytes(100_000, 300) == 2 * 100_000 * 300 * 8
    assert w2v.step_batch_workspace_bytes(3, 5) == 2 * 256
    assert w2v.step_batch_workspace_bytes(0, 5) == 0
    # two matrices x split rows x 8 partial rows x ld floats
    assert w2v.train_epoch_workspace_bytes(3, 300) == 2 * 3 * 8 * 300 * 4
    assert w2v.train_epoch_workspace_bytes(0, 300) == 0


def test_hot_rows_model():
    """Uniform counts: every word has the same write rate, so either all rows
    or none are hot; the count grows with the number in flight."""
    V = 1000
    counts = np.full(V, 10, np.int64)
    # rho = 1/V, q = 1/V -> p = max(rho + K q, (w+1) rho) = 6/V with K=5, w=5
    p = 6.0 / V
    assert w2v.hot_rows(counts, sample_t=0.0, inflight=int(0.5 / p) + 2, tol=0.5) == V
    assert w2v.hot_rows(counts, sample_t=0.0, inflight=int(0.5 / p) - 1, tol=0.5) == 0
    zipf = np.rint(inputs.zipf_pmf(100_000, 1.07) * 1e8).astype(np.int64)
    hs = [w2v.hot_rows(zipf, inflight=f) for f in (16, 256, 4096)]
    assert hs[0] < hs[1] < hs[2] < 100_000
    assert w2v.hot_rows(zipf, inflight=256, tol=0.5) < hs[1]   # default tol 0.05


def test_hot_rows_rejects():
    c = np.ones(4, np.int64)
    for kw in (dict(inflight=0), dict(tol=0.0), dict(window=0), dict(K=-1)):
        args = dict(inflight=10)
        args.update(kw)
        with pytest.raises(w2v.W2VError):
            w2v.hot_rows(c, **args)


def vocab(**over):
    args = dict(raw=FAKE, T=100, V=10, min_count=0, ranked=FAKE, rank_of=FAKE,
                v_kept=FAKE, corpus=None, ws=0x100000, ws_bytes=1 << 20, stream=None)
    args.update(over)
    return w2v.lib().w2v_build_vocab(*args.values())


@pytest.mark.parametrize("over,needle", [
    (dict(T=-1), "T"), (dict(raw=None), "raw"), (dict(V=0), "V_raw"),
    (dict(min_count=-1), "min_count"), (dict(ranked=None), "NULL"),
    (dict(v_kept=None), "NULL"), (dict(ws=None), "workspace"),
    (dict(ws_bytes=10), "workspace"), (dict(ws=0x100008), "aligned"),
])
def test_build_vocab_rejects(over, needle):
    assert vocab(**over) == w2v.EINVAL
    assert needle in w2v.lib().w2v_last_error().decode()


def test_build_vocab_workspace_sizes():
    """Up to 4,194,304 raw ids the ids are counted by bins, whose workspace
    holds the binned corpus (at least 4 bytes per token); above, the count
    needs no T-sized workspace."""
    ws = w2v.lib().w2v_build_vocab_workspace_bytes
    assert ws(0, 10) == 0 and ws(10, -1) == 0
    for V in (1, 32768, 32769, 2_000_000, 4_194_304):
        assert ws(V, 10**6) - ws(V, 0) >= 4 * 10**6
        assert ws(V, 10**7) - ws(V, 10**6) >= 4 * 9 * 10**6
    assert ws(4_194_305, 10**7) == ws(4_194_305, 0)


@pytest.mark.parametrize("args,needle", [
    ((0, 5, 5), "D"), ((641, 5, 5), "D"), ((300, 0, 5), "window"),
    ((300, 17, 5), "window"), ((300, 5, -1), "K"), ((300, 5, 65), "K"),
])
def test_pending_slots_rejects(args, needle):
    assert w2v.lib().w2v_pending_slots(*args) == w2v.EINVAL
    assert needle in w2v.lib().w2v_last_error().decode()


def sorted_step(**over):
    args = dict(B=4, N=2, K=1, t=FAKE, c=FAKE, n=FAKE, alpha=None, a_s=0.0,
                Mi=FAKE, Mo=FAKE + 0x1000, V=10, D=8, ld=8, ws=0x100000,
                ws_bytes=1 << 30, stats=None, stream=None)
    args.update(over)
    return w2v.lib().w2v_step_batch_sorted(*args.values())


@pytest.mark.parametrize("over,needle", [
    (dict(B=-1), "B"), (dict(N=33), "N"), (dict(K=65), "K"),
    (dict(B=1 << 30, K=64), "int32"), (dict(t=None), "targets"),
    (dict(c=None), "contexts"), (dict(n=None), "negatives"), (dict(D=9), "D"),
])
def test_step_batch_sorted_rejects(over, needle):
    assert sorted_step(**over) == w2v.EINVAL
    assert needle in w2v.lib().w2v_last_error().decode()


def test_step_batch_sorted_workspace_rejects_invalid_shapes():
    L = w2v.lib()
    for args in ((-1, 2, 1, 10, 8), (4, -1, 1, 10, 8), (4, 2, -1, 10, 8),
                 (4, 2, 1, 0, 8), (4, 2, 1, 10, 0)):
        assert L.w2v_step_batch_sorted_workspace_bytes(*args) == 0


def test_check_loss_rejects():
    L = w2v.lib()
    assert L.w2v_check_loss(None, -1, None) == w2v.EINVAL
    assert "n_buckets" in L.w2v_last_error().decode()
    assert L.w2v_check_loss(None, 3, None) == w2v.EINVAL
    assert "NULL" in L.w2v_last_error().decode()
