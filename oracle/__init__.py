"""CPU oracle for the HogBatch SGNS step (Ji et al., arXiv 1611.06172).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg load it; the GPU library never does. This module is a thin
ctypes loader over the plain C oracle in this directory (fp64 arithmetic, one
thread); numpy arrays in, numpy arrays out. It imports nothing from the GPU
package.
"""
import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_u32p = ctypes.POINTER(ctypes.c_uint32)
_u64p = ctypes.POINTER(ctypes.c_uint64)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)


class _Sampling(ctypes.Structure):
    _fields_ = [
        ("corpus", _i32p), ("T", ctypes.c_int64),
        ("pos_begin", ctypes.c_int64), ("pos_end", ctypes.c_int64),
        ("sentence_len", ctypes.c_int32), ("window", ctypes.c_int32),
        ("K", ctypes.c_int32), ("neg_table", _i32p),
        ("table_size", ctypes.c_int64), ("keep_thresh", _u32p),
        ("alpha0", ctypes.c_float), ("min_alpha_frac", ctypes.c_float),
        ("epoch", ctypes.c_int32), ("n_epochs", ctypes.c_int32),
        ("seed", ctypes.c_uint64),
    ]


def lib():
    """Loads liboracle.so, building it first when it is absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _build
            _build.build()
        L = ctypes.CDLL(_LIB_PATH)
        L.oracle_philox4x64_10.argtypes = [_u64p, _u64p, _u64p]
        L.oracle_philox4x64_10.restype = None
        L.oracle_draw_u32.argtypes = [ctypes.c_uint64] * 3 + [ctypes.c_uint32]
        L.oracle_draw_u32.restype = ctypes.c_uint32
        L.oracle_build_tables.argtypes = [_i64p, ctypes.c_int32, ctypes.c_double,
                                          ctypes.c_double, _i32p, ctypes.c_int64,
                                          _u32p]
        L.oracle_build_tables.restype = ctypes.c_int
        L.oracle_minibatches.argtypes = [ctypes.POINTER(_Sampling), _i32p, _i32p,
                                         _i32p, _u8p, _f32p, _i64p, ctypes.c_int64]
        L.oracle_minibatches.restype = ctypes.c_int64
        L.oracle_sgns_delta.argtypes = [ctypes.c_int32] * 3 + [_f64p, _f64p, _u8p,
                                        ctypes.c_double, _f64p, _f64p, _f64p, _f64p]
        L.oracle_sgns_delta.restype = None
        L.oracle_sgns_delta_scaled.argtypes = [ctypes.c_int32] * 3 + [
            _f64p, _f64p, _u8p, ctypes.c_double, _f64p, _f64p, _f64p, _f64p,
            _f64p, _f64p]
        L.oracle_sgns_delta_scaled.restype = None
        L.oracle_apply_minibatch.argtypes = [
            _f32p, _f32p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
            ctypes.c_int32, _i32p, ctypes.c_int32, ctypes.c_int32, _i32p, _u8p,
            ctypes.c_float, _f64p, _i32p]
        L.oracle_apply_minibatch.restype = ctypes.c_int
        L.oracle_step_batch.argtypes = [
            ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _i32p, _i32p, _i32p,
            _f32p, ctypes.c_float, _f32p, _f32p, ctypes.c_int32, ctypes.c_int32,
            ctypes.c_int32, _f64p, _f64p]
        L.oracle_step_batch.restype = ctypes.c_int
        L.oracle_train_epoch.argtypes = [ctypes.POINTER(_Sampling), _f32p, _f32p,
                                         ctypes.c_int32, ctypes.c_int32,
                                         ctypes.c_int32, _f64p, ctypes.c_int32]
        L.oracle_train_epoch.restype = ctypes.c_int64
        L.oracle_pair_negative.argtypes = [ctypes.POINTER(_Sampling), ctypes.c_int64,
                                           ctypes.c_int32, ctypes.c_int32]
        L.oracle_pair_negative.restype = ctypes.c_int32
        L.oracle_pairwise_train_epoch.argtypes = [ctypes.POINTER(_Sampling), _f32p,
                                                  _f32p, ctypes.c_int32, ctypes.c_int32,
                                                  ctypes.c_int32, _f64p, ctypes.c_int32]
        L.oracle_pairwise_train_epoch.restype = ctypes.c_int64
        L.oracle_grouped_train_epoch.argtypes = [ctypes.POINTER(_Sampling), ctypes.c_int32,
                                                 _f32p, _f32p, ctypes.c_int32,
                                                 ctypes.c_int32, ctypes.c_int32, _f64p,
                                                 ctypes.c_int32]
        L.oracle_grouped_train_epoch.restype = ctypes.c_int64
        _lib = L
    return _lib


def _ptr(a, ctype):
    if a is None:
        return None
    return a.ctypes.data_as(ctype)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def philox4x64_10(ctr, key):
    """One Philox4x64-10 block: counter (4 x u64), key (2 x u64) -> 4 x u64."""
    c = _c(ctr, np.uint64)
    k = _c(key, np.uint64)
    out = np.zeros(4, dtype=np.uint64)
    lib().oracle_philox4x64_10(_ptr(c, _u64p), _ptr(k, _u64p), _ptr(out, _u64p))
    return out


def draw_u32(seed: int, p: int, e: int, word: int) -> int:
    """Word `word` of the random stream of raw position p in epoch e."""
    return int(lib().oracle_draw_u32(seed, p, e, word))


def build_tables(counts, neg_power=0.75, sample_t=1e-4, table_size=10**8,
                 want_table=True, want_thresh=True):
    """Negative table (int32[table_size]) and keep thresholds (uint32[V])."""
    counts = _c(counts, np.int64)
    V = counts.shape[0]
    table = np.empty(table_size, dtype=np.int32) if want_table else None
    thresh = np.empty(V, dtype=np.uint32) if want_thresh else None
    rc = lib().oracle_build_tables(_ptr(counts, _i64p), V, neg_power, sample_t,
                                   _ptr(table, _i32p), table_size,
                                   _ptr(thresh, _u32p))
    if rc != 0:
        raise ValueError(f"oracle_build_tables failed ({rc})")
    return table, thresh


@dataclass
class Sampling:
    """Sampling configuration of one epoch (or a sentence-aligned range)."""
    corpus: np.ndarray
    neg_table: np.ndarray
    keep_thresh: Optional[np.ndarray]
    window: int = 5
    K: int = 5
    sentence_len: int = 1000
    alpha0: float = 0.025
    min_alpha_frac: float = 1e-4
    epoch: int = 0
    n_epochs: int = 1
    seed: int = 0
    pos_begin: int = 0
    pos_end: Optional[int] = None

    def _struct(self):
        self._keep = [_c(self.corpus, np.int32), _c(self.neg_table, np.int32),
                      None if self.keep_thresh is None
                      else _c(self.keep_thresh, np.uint32)]
        corpus, table, thr = self._keep
        T = corpus.shape[0]
        end = T if self.pos_end is None else self.pos_end
        return _Sampling(_ptr(corpus, _i32p), T, self.pos_begin, end,
                         self.sentence_len, self.window, self.K,
                         _ptr(table, _i32p), table.shape[0], _ptr(thr, _u32p),
                         self.alpha0, self.min_alpha_frac, self.epoch,
                         self.n_epochs, self.seed)


def minibatches(s: Sampling):
    """All minibatches of the range, in processing order, as a dict of arrays."""
    st = s._struct()
    L = lib()
    n = L.oracle_minibatches(ctypes.byref(st), None, None, None, None, None,
                             None, 0)
    if n < 0:
        raise ValueError("oracle_minibatches: bad arguments")
    w2 = 2 * s.window
    out = dict(targets=np.empty(n, np.int32), ctx=np.empty((n, w2), np.int32),
               negs=np.empty((n, s.K), np.int32), mask=np.empty((n, s.K), np.uint8),
               alpha=np.empty(n, np.float32), pos=np.empty(n, np.int64))
    m = L.oracle_minibatches(ctypes.byref(st), _ptr(out["targets"], _i32p),
                             _ptr(out["ctx"], _i32p), _ptr(out["negs"], _i32p),
                             _ptr(out["mask"], _u8p), _ptr(out["alpha"], _f32p),
                             _ptr(out["pos"], _i64p), n)
    assert m == n
    return out


def sgns_delta(A, O, mask, alpha):
    """fp64 minibatch maths: returns (X, dA, dO, loss)."""
    A = _c(A, np.float64)
    O = _c(O, np.float64)
    N, D = A.shape
    K = O.shape[0] - 1
    mask = _c(mask if mask is not None else np.zeros(K, np.uint8), np.uint8)
    X = np.empty((N, K + 1))
    dA = np.empty((N, D))
    dO = np.empty((K + 1, D))
    loss = ctypes.c_double()
    lib().oracle_sgns_delta(N, K, D, _ptr(A, _f64p), _ptr(O, _f64p),
                            _ptr(mask, _u8p), float(alpha), _ptr(X, _f64p),
                            _ptr(dA, _f64p), _ptr(dO, _f64p), ctypes.byref(loss))
    return X, dA, dO, loss.value


def sgns_delta_scaled(A, O, mask, alpha):
    """sgns_delta plus the per-element error scales: (X, dA, dO, loss, sA, sO)
    with sA = |E| |O| and sO = |E|^T |A|."""
    A = _c(A, np.float64)
    O = _c(O, np.float64)
    N, D = A.shape
    K = O.shape[0] - 1
    mask = _c(mask if mask is not None else np.zeros(K, np.uint8), np.uint8)
    X = np.empty((N, K + 1))
    dA = np.empty((N, D))
    dO = np.empty((K + 1, D))
    sA = np.empty((N, D))
    sO = np.empty((K + 1, D))
    loss = ctypes.c_double()
    lib().oracle_sgns_delta_scaled(N, K, D, _ptr(A, _f64p), _ptr(O, _f64p),
                                   _ptr(mask, _u8p), float(alpha), _ptr(X, _f64p),
                                   _ptr(dA, _f64p), _ptr(dO, _f64p),
                                   ctypes.byref(loss), _ptr(sA, _f64p),
                                   _ptr(sO, _f64p))
    return X, dA, dO, loss.value, sA, sO


def apply_minibatch(M_in, M_out, ctx, target, negs, alpha, mask=None):
    """Applies one minibatch in place to fp32 matrices; returns (loss, n_ctx)."""
    assert M_in.dtype == np.float32 and M_in.flags.c_contiguous
    assert M_out.dtype == np.float32 and M_out.flags.c_contiguous
    V, ld = M_in.shape
    ctx = _c(ctx, np.int32)
    negs = _c(negs, np.int32)
    K = negs.shape[0]
    if mask is None:
        mask = (negs == target).astype(np.uint8)
    mask = _c(mask, np.uint8)
    loss = ctypes.c_double()
    n = ctypes.c_int32()
    rc = lib().oracle_apply_minibatch(
        _ptr(M_in, _f32p), _ptr(M_out, _f32p), V, ld, ld, ctx.shape[0],
        _ptr(ctx, _i32p), int(target), K, _ptr(negs, _i32p), _ptr(mask, _u8p),
        float(alpha), ctypes.byref(loss), ctypes.byref(n))
    if rc != 0:
        raise ValueError(f"oracle_apply_minibatch failed ({rc})")
    return loss.value, n.value


def step_batch(targets, contexts, negatives, M_in, M_out, alpha=0.025,
               D=None, with_scale=True):
    """Snapshot batch: returns (M_in', M_out', S_in, S_out) as new arrays.

    alpha is a scalar or an array of B learning rates. S_* are the per-element
    error scales |M0| + sum over occurrences of sum |products| (None when
    with_scale is False).
    """
    targets = _c(targets, np.int32)
    contexts = _c(contexts, np.int32)
    negatives = _c(negatives, np.int32)
    B = targets.shape[0]
    N = contexts.shape[1] if contexts.ndim == 2 else 0
    K = negatives.shape[1] if negatives.ndim == 2 else 0
    Mi = np.array(M_in, dtype=np.float32, copy=True, order="C")
    Mo = np.array(M_out, dtype=np.float32, copy=True, order="C")
    V, ld = Mi.shape
    D = ld if D is None else D
    S_in = np.empty((V, D)) if with_scale else None
    S_out = np.empty((V, D)) if with_scale else None
    if np.ndim(alpha) == 0:
        a_arr, a_s = None, float(alpha)
    else:
        a_arr, a_s = _c(alpha, np.float32), 0.0
    rc = lib().oracle_step_batch(B, N, K, _ptr(targets, _i32p),
                                 _ptr(contexts, _i32p), _ptr(negatives, _i32p),
                                 _ptr(a_arr, _f32p), a_s, _ptr(Mi, _f32p),
                                 _ptr(Mo, _f32p), V, D, ld, _ptr(S_in, _f64p),
                                 _ptr(S_out, _f64p))
    if rc != 0:
        raise ValueError(f"oracle_step_batch failed ({rc})")
    return Mi, Mo, S_in, S_out


def train_epoch(s: Sampling, M_in, M_out, D=None, n_buckets=0):
    """Sequential epoch, in place on fp32 matrices.

    Returns (minibatches applied, loss_buckets[n_buckets, 2] or None).
    """
    assert M_in.dtype == np.float32 and M_in.flags.c_contiguous
    assert M_out.dtype == np.float32 and M_out.flags.c_contiguous
    V, ld = M_in.shape
    D = ld if D is None else D
    st = s._struct()
    buckets = np.zeros((n_buckets, 2)) if n_buckets > 0 else None
    n = lib().oracle_train_epoch(ctypes.byref(st), _ptr(M_in, _f32p),
                                 _ptr(M_out, _f32p), V, D, ld,
                                 _ptr(buckets, _f64p), n_buckets)
    if n < 0:
        raise ValueError("oracle_train_epoch failed")
    return n, buckets


def pair_negatives(s: Sampling, p: int, n_inputs: int) -> np.ndarray:
    """[n_inputs, K] negatives of Algorithm 1 for the target at raw position
    p: row i holds the K draws of input word i."""
    st = s._struct()
    out = np.empty((n_inputs, s.K), dtype=np.int32)
    for i in range(n_inputs):
        for k in range(s.K):
            out[i, k] = lib().oracle_pair_negative(ctypes.byref(st), p, i, k)
    return out


def pairwise_train_epoch(s: Sampling, M_in, M_out, D=None, n_buckets=0):
    """Algorithm 1 (per-pair Hogwild SGD), sequential, in place on fp32
    matrices. Returns (targets applied, loss_buckets[n_buckets, 2] or None)."""
    assert M_in.dtype == np.float32 and M_in.flags.c_contiguous
    assert M_out.dtype == np.float32 and M_out.flags.c_contiguous
    V, ld = M_in.shape
    D = ld if D is None else D
    st = s._struct()
    buckets = np.zeros((n_buckets, 2)) if n_buckets > 0 else None
    n = lib().oracle_pairwise_train_epoch(ctypes.byref(st), _ptr(M_in, _f32p),
                                          _ptr(M_out, _f32p), V, D, ld,
                                          _ptr(buckets, _f64p), n_buckets)
    if n < 0:
        raise ValueError("oracle_pairwise_train_epoch failed")
    return n, buckets


def grouped_train_epoch(s: Sampling, G: int, M_in, M_out, D=None, n_buckets=0):
    """HogBatch with negatives shared by groups of G consecutive targets,
    sequential, in place. Returns (minibatches applied, loss buckets)."""
    assert M_in.dtype == np.float32 and M_in.flags.c_contiguous
    assert M_out.dtype == np.float32 and M_out.flags.c_contiguous
    V, ld = M_in.shape
    D = ld if D is None else D
    st = s._struct()
    buckets = np.zeros((n_buckets, 2)) if n_buckets > 0 else None
    n = lib().oracle_grouped_train_epoch(ctypes.byref(st), G, _ptr(M_in, _f32p),
                                         _ptr(M_out, _f32p), V, D, ld,
                                         _ptr(buckets, _f64p), n_buckets)
    if n < 0:
        raise ValueError("oracle_grouped_train_epoch failed")
    return n, buckets


from .vocab import build_vocab  # noqa: E402,F401  (numpy-only reference)
