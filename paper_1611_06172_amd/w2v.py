"""ctypes binding of libw2v (include/w2v.h): argument marshalling only.

Every function takes torch tensors that already live where the C ABI expects
them (device tensors on the current HIP device for GPU entry points), checks
dtypes and shapes, and passes raw pointers plus the current torch stream.
No arithmetic of the method happens here. If libw2v.so has not been built the
first call raises: there is no CPU fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libw2v.so")

_vp = ctypes.c_void_p
_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_f32 = ctypes.c_float
_f64 = ctypes.c_double
_u64 = ctypes.c_uint64

_lib = None

OK = 0
EINVAL = -1
EHIP = -2
ENOMEM = -3
EUNSUPPORTED = -4
EDEVICE_FLAG = -5
ENONFINITE = -6


class W2VError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libw2v error {code}: {msg}")
        self.code = code


def lib():
    """The loaded libw2v.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
            "(hipcc, gfx950) before using the GPU path")
    L = ctypes.CDLL(LIB_PATH)
    L.w2v_version.restype = ctypes.c_int
    L.w2v_last_error.restype = ctypes.c_char_p
    L.w2v_init.argtypes = []
    L.w2v_init.restype = ctypes.c_int
    L.w2v_device_status.argtypes = [_vp]
    L.w2v_device_status.restype = ctypes.c_int
    L.w2v_check_loss.argtypes = [_vp, _i32, _vp]
    L.w2v_check_loss.restype = ctypes.c_int
    L.w2v_build_tables.argtypes = [_vp, _i32, _f64, _f64, _vp, _i64, _vp]
    L.w2v_build_tables.restype = ctypes.c_int
    L.w2v_train_epoch.argtypes = [
        _vp, _i64, _i64, _i64, _i32, _vp, _vp, _i32, _i32, _i32, _i32, _i32,
        _vp, _i64, _vp, _f32, _f32, _i32, _i32, _u64, _vp, _i32, _vp, _i32, _i32,
        _i32, _vp, ctypes.c_size_t, _i32, _i32, _vp]
    L.w2v_train_epoch.restype = ctypes.c_int
    L.w2v_train_epoch_noalloc.argtypes = (L.w2v_train_epoch.argtypes[:26] +
                                          L.w2v_train_epoch.argtypes[28:])
    L.w2v_train_epoch_noalloc.restype = ctypes.c_int
    L.w2v_build_vocab_workspace_bytes.argtypes = [_i32, _i64]
    L.w2v_build_vocab_workspace_bytes.restype = ctypes.c_size_t
    L.w2v_build_vocab.argtypes = [_vp, _i64, _i32, _i64, _vp, _vp, _vp, _vp, _vp,
                                  ctypes.c_size_t, _vp]
    L.w2v_build_vocab.restype = ctypes.c_int
    L.w2v_train_epoch_workspace_bytes.argtypes = [_i32, _i32]
    L.w2v_train_epoch_workspace_bytes.restype = ctypes.c_size_t
    L.w2v_debug_minibatches.argtypes = [
        _vp, _i64, _i64, _i64, _i32, _i32, _i32, _i32, _vp, _i64, _vp, _f32,
        _f32, _i32, _i32, _u64, _vp, _vp, _vp, _vp, _vp, _vp, _vp]
    L.w2v_debug_minibatches.restype = ctypes.c_int
    L.w2v_hot_rows.argtypes = [_vp, _i32, _f64, _f64, _i32, _i32, _i64, _f64]
    L.w2v_hot_rows.restype = ctypes.c_int32
    L.w2v_default_inflight.argtypes = [_i32, _i32, _i32, _i32, _i32]
    L.w2v_default_inflight.restype = ctypes.c_int64
    L.w2v_pending_slots.argtypes = [_i32, _i32, _i32]
    L.w2v_pending_slots.restype = ctypes.c_int32
    L.w2v_step_batch_workspace_bytes.argtypes = [_i32, _i32]
    L.w2v_step_batch_workspace_bytes.restype = ctypes.c_size_t
    L.w2v_step_batch.argtypes = [
        _i32, _i32, _i32, _vp, _vp, _vp, _vp, _f32, _vp, _vp, _i32, _i32, _i32,
        _vp, ctypes.c_size_t, _vp, _vp]
    L.w2v_step_batch.restype = ctypes.c_int
    L.w2v_step_batch_sorted_workspace_bytes.argtypes = [_i32, _i32, _i32, _i32, _i32]
    L.w2v_step_batch_sorted_workspace_bytes.restype = ctypes.c_size_t
    L.w2v_step_batch_sorted.argtypes = L.w2v_step_batch.argtypes
    L.w2v_step_batch_sorted.restype = ctypes.c_int
    _lib = L
    return L


def _check(rc: int):
    if rc != OK:
        raise W2VError(rc, lib().w2v_last_error().decode())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    return t.data_ptr()


def _stream(stream=None) -> int:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _dev(t, dtype, name, ndim=None):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if isinstance(dtype, tuple):
        if t.dtype not in dtype:
            raise TypeError(f"{name} must have dtype in {dtype}, got {t.dtype}")
    elif t.dtype != dtype:
        raise TypeError(f"{name} must have dtype {dtype}, got {t.dtype}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must be {ndim}-D")
    # The kernels index every argument but the two matrices as packed arrays
    # (contexts[b N + i], loss[2 b], ...): a strided view would be read at
    # the wrong places, so only contiguous tensors pass.
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _matrix(M, name):
    """Checks a V x D fp32 device matrix; rows may be padded (the row stride
    is passed to the library as ld), columns must be adjacent."""
    import torch
    if not isinstance(M, torch.Tensor) or not M.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if M.dtype != torch.float32:
        raise TypeError(f"{name} must have dtype torch.float32, got {M.dtype}")
    if M.dim() != 2:
        raise ValueError(f"{name} must be 2-D")
    if M.stride(1) != 1 or M.stride(0) < M.shape[1]:
        raise ValueError(f"{name} must have unit column stride and a row stride >= D")
    return M.shape[0], M.stride(0)


def version() -> int:
    return int(lib().w2v_version())


def build_tables(counts, neg_power: float = 0.75, sample_t: float = 1e-4,
                 table_size: int = 10**8, want_table: bool = True,
                 want_thresh: bool = True):
    """Host tables: (neg_table int32[table_size], keep_thresh uint32[V])."""
    counts = np.ascontiguousarray(counts, dtype=np.int64)
    V = counts.shape[0]
    table = np.empty(table_size, dtype=np.int32) if want_table else None
    thr = np.empty(V, dtype=np.uint32) if want_thresh else None
    _check(lib().w2v_build_tables(
        counts.ctypes.data, V, float(neg_power), float(sample_t),
        None if table is None else table.ctypes.data, int(table_size),
        None if thr is None else thr.ctypes.data))
    return table, thr


def hot_rows(counts, *, neg_power: float = 0.75, sample_t: float = 1e-4,
             window: int = 5, K: int = 5, inflight: int, tol: float = 0.05) -> int:
    """Leading ids to update atomically (see w2v_hot_rows). The default
    tolerance keeps the expected share of overwritten updates of a plain row
    near 5% (1 - exp(-tol))."""
    counts = np.ascontiguousarray(counts, dtype=np.int64)
    h = int(lib().w2v_hot_rows(counts.ctypes.data, counts.shape[0],
                                float(neg_power), float(sample_t), window, K,
                                int(inflight), float(tol)))
    if h < 0:
        _check(h)
    return h


def init():
    """Sets up the library's state on the current device (w2v_init)."""
    _check(lib().w2v_init())


def device_status(stream=None):
    """Waits for the stream, then raises W2VError (code EDEVICE_FLAG) if a
    kernel of the library skipped work for an id outside [0, V) since this
    was last reported (w2v_device_status)."""
    _check(lib().w2v_device_status(_stream(stream)))


def check_loss(loss_buckets, stream=None):
    """Waits for the stream, then raises W2VError (code ENONFINITE) naming the
    first loss bucket whose sum or count is NaN or Inf (w2v_check_loss)."""
    import torch
    _dev(loss_buckets, torch.float64, "loss_buckets", 2)
    _check(lib().w2v_check_loss(_ptr(loss_buckets), loss_buckets.shape[0],
                                _stream(stream)))


def default_inflight(D: int, window: int = 5, K: int = 5, *, V: int,
                     group: int = 1) -> int:
    """Concurrent sentences of train_epoch with max_inflight = 0 over a
    vocabulary of V words (w2v_default_inflight)."""
    n = int(lib().w2v_default_inflight(V, D, window, K, group))
    if n < 0:
        _check(n)
    return n


def pending_slots(D: int, window: int = 5, K: int = 5) -> int:
    """LDS slots per wavefront in which HogBatch training collects pending
    updates of cold input rows (0: none)."""
    n = int(lib().w2v_pending_slots(D, window, K))
    if n < 0:
        _check(n)
    return n


ALGORITHMS = {"hogbatch": 0, "pairwise": 1, "hogbatch_immediate": 2}


def train_epoch(corpus, M_in, M_out, neg_table, keep_thresh=None, *,
                window: int = 5, K: int = 5, D: Optional[int] = None,
                alpha0: float = 0.025, min_alpha_frac: float = 1e-4,
                epoch: int = 0, n_epochs: int = 1, seed: int = 0,
                pos_begin: int = 0, pos_end: Optional[int] = None,
                sentence_len: int = 1000, loss_buckets=None, stats=None,
                max_inflight: int = 0, hot_rows: Optional[int] = None,
                split_rows: int = 0, workspace=None, algorithm: str = "hogbatch",
                group: int = 1, stream=None):
    """Hogwild HogBatch epoch over corpus[pos_begin:pos_end], in place.

    hot_rows: ids below it are updated with atomic adds, the others with
    plain read-modify-write stores; None makes every update atomic.
    split_rows: ids below it are updated through per-XCD partial rows that
    every read sums (see w2v_train_epoch); workspace (a device byte tensor of
    train_epoch_workspace_bytes(split_rows, ld)) is allocated when None.
    algorithm: "hogbatch" (Sec. 1.1; cold input rows collect their updates
        in LDS while their word is in the window, see w2v_train_epoch),
        "hogbatch_immediate" (every update applied at the end of its
        minibatch) or "pairwise" (Alg. 1, the baseline).
    group: consecutive targets sharing one draw of negatives (1: HogBatch as
    in the paper; 2, 4, 8: the sharing widened across targets)."""
    import torch
    _dev(corpus, torch.int32, "corpus", 1)
    V, ld = _matrix(M_in, "M_in")
    V2, ld2 = _matrix(M_out, "M_out")
    if (V, ld) != (V2, ld2):
        raise ValueError("M_in and M_out must have the same shape and stride")
    D = M_in.shape[1] if D is None else D
    _dev(neg_table, torch.int32, "neg_table", 1)
    if keep_thresh is not None:
        _dev(keep_thresh, (torch.int32, torch.uint32), "keep_thresh", 1)
        if keep_thresh.numel() != V:
            raise ValueError("keep_thresh must have V entries")
    n_b = 0
    if loss_buckets is not None:
        _dev(loss_buckets, torch.float64, "loss_buckets", 2)
        n_b = loss_buckets.shape[0]
    if stats is not None:
        _dev(stats, torch.int64, "stats", 1)
        if stats.numel() < 5:
            raise ValueError("stats must have 5 entries (see w2v_train_epoch)")
    T = corpus.numel()
    end = T if pos_end is None else pos_end
    need = train_epoch_workspace_bytes(split_rows, ld)
    if need and workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=M_in.device)
    ws_bytes = 0
    if workspace is not None:
        _dev(workspace, torch.uint8, "workspace", 1)
        ws_bytes = workspace.numel()
    _check(lib().w2v_train_epoch(
        _ptr(corpus), T, pos_begin, end, sentence_len, _ptr(M_in), _ptr(M_out),
        V, D, ld, window, K, _ptr(neg_table), neg_table.numel(),
        _ptr(keep_thresh), alpha0, min_alpha_frac, epoch, n_epochs, seed,
        _ptr(loss_buckets), n_b, _ptr(stats), max_inflight,
        V if hot_rows is None else int(hot_rows), int(split_rows),
        _ptr(workspace), ws_bytes, ALGORITHMS[algorithm], int(group),
        _stream(stream)))


NOALLOC_SCRATCH_BYTES = 4194304


def train_epoch_noalloc(corpus, M_in, M_out, neg_table, keep_thresh=None, *,
                        window: int = 5, K: int = 5, D: Optional[int] = None,
                        alpha0: float = 0.025, min_alpha_frac: float = 1e-4,
                        epoch: int = 0, n_epochs: int = 1, seed: int = 0,
                        pos_begin: int = 0, pos_end: Optional[int] = None,
                        sentence_len: int = 1000, loss_buckets=None, stats=None,
                        max_inflight: int = 0, hot_rows: Optional[int] = None,
                        split_rows: int = 0, algorithm: str = "hogbatch",
                        group: int = 1, stream=None):
    """train_epoch through w2v_train_epoch_noalloc: the split rows' partial
    rows live in the library's static device scratch array, so nothing is
    allocated here or in the library. init() must have run on the device."""
    import torch
    _dev(corpus, torch.int32, "corpus", 1)
    V, ld = _matrix(M_in, "M_in")
    if _matrix(M_out, "M_out") != (V, ld):
        raise ValueError("M_in and M_out must have the same shape and stride")
    D = M_in.shape[1] if D is None else D
    _dev(neg_table, torch.int32, "neg_table", 1)
    if keep_thresh is not None:
        _dev(keep_thresh, (torch.int32, torch.uint32), "keep_thresh", 1)
        if keep_thresh.numel() != V:
            raise ValueError("keep_thresh must have V entries")
    n_b = 0
    if loss_buckets is not None:
        _dev(loss_buckets, torch.float64, "loss_buckets", 2)
        n_b = loss_buckets.shape[0]
    if stats is not None:
        _dev(stats, torch.int64, "stats", 1)
        if stats.numel() < 5:
            raise ValueError("stats must have 5 entries (see w2v_train_epoch)")
    T = corpus.numel()
    end = T if pos_end is None else pos_end
    _check(lib().w2v_train_epoch_noalloc(
        _ptr(corpus), T, pos_begin, end, sentence_len, _ptr(M_in), _ptr(M_out),
        V, D, ld, window, K, _ptr(neg_table), neg_table.numel(),
        _ptr(keep_thresh), alpha0, min_alpha_frac, epoch, n_epochs, seed,
        _ptr(loss_buckets), n_b, _ptr(stats), max_inflight,
        V if hot_rows is None else int(hot_rows), int(split_rows),
        ALGORITHMS[algorithm], int(group), _stream(stream)))


def padded_ld(D: int) -> int:
    """Row stride (floats) that starts every row on a 128-byte line: D
    rounded up to a multiple of 32."""
    return (D + 31) // 32 * 32


def alloc_matrix(V: int, D: int, device="cuda", init=None):
    """A (V, D) fp32 view of a zeroed (V, padded_ld(D)) device buffer,
    optionally filled from `init` (array-like of shape (V, D)). Line-aligned
    rows cost fewer partial-line reads and writes than a packed (V, D)
    matrix when rows are gathered and scattered at random."""
    import torch
    buf = torch.zeros((V, padded_ld(D)), dtype=torch.float32, device=device)
    M = buf[:, :D]
    if init is not None:
        M.copy_(torch.as_tensor(init))
    return M


def train_epoch_workspace_bytes(split_rows: int, ld: int) -> int:
    return int(lib().w2v_train_epoch_workspace_bytes(split_rows, ld))


def debug_minibatches(corpus, neg_table, keep_thresh=None, *, V: int,
                      window: int = 5, K: int = 5, alpha0: float = 0.025,
                      min_alpha_frac: float = 1e-4, epoch: int = 0,
                      n_epochs: int = 1, seed: int = 0, pos_begin: int = 0,
                      pos_end: Optional[int] = None, sentence_len: int = 1000,
                      stats=None, stream=None):
    """Minibatches the epoch would form, indexed by raw position (GPU)."""
    import torch
    _dev(corpus, torch.int32, "corpus", 1)
    _dev(neg_table, torch.int32, "neg_table", 1)
    if keep_thresh is not None:
        _dev(keep_thresh, (torch.int32, torch.uint32), "keep_thresh", 1)
    if stats is not None:
        _dev(stats, torch.int64, "stats", 1)
        if stats.numel() < 5:
            raise ValueError("stats must have 5 entries (see w2v_train_epoch)")
    T = corpus.numel()
    end = T if pos_end is None else pos_end
    P = end - pos_begin
    dev = corpus.device
    out = dict(
        targets=torch.empty(P, dtype=torch.int32, device=dev),
        ctx=torch.empty((P, 2 * window), dtype=torch.int32, device=dev),
        negs=torch.empty((P, K), dtype=torch.int32, device=dev),
        mask=torch.empty((P, K), dtype=torch.uint8, device=dev),
        alpha=torch.empty(P, dtype=torch.float32, device=dev))
    _check(lib().w2v_debug_minibatches(
        _ptr(corpus), T, pos_begin, end, sentence_len, V, window, K,
        _ptr(neg_table), neg_table.numel(), _ptr(keep_thresh), alpha0,
        min_alpha_frac, epoch, n_epochs, seed, _ptr(out["targets"]),
        _ptr(out["ctx"]), _ptr(out["negs"]), _ptr(out["mask"]),
        _ptr(out["alpha"]), _ptr(stats), _stream(stream)))
    return out


def step_batch_workspace_bytes(V: int, ld: int) -> int:
    return int(lib().w2v_step_batch_workspace_bytes(V, ld))


def alloc_workspace(V: int, ld: int, device="cuda"):
    """A torch-owned byte buffer large enough for step_batch."""
    import torch
    n = step_batch_workspace_bytes(V, ld)
    return torch.empty(n, dtype=torch.uint8, device=device)


def step_batch_sorted_workspace_bytes(B: int, N: int, K: int, V: int, ld: int) -> int:
    return int(lib().w2v_step_batch_sorted_workspace_bytes(B, N, K, V, ld))


def step_batch(targets, contexts, negatives, M_in, M_out, alpha=0.025, *,
               D: Optional[int] = None, workspace=None, stats=None,
               stream=None, sorted: bool = False):
    """One snapshot batch of B minibatches; updates M_in, M_out in place.
    sorted: sum each row's updates in a fixed order (w2v_step_batch_sorted:
    the same bits on every run) instead of with fp64 atomics."""
    import torch
    _dev(targets, torch.int32, "targets", 1)
    _dev(contexts, torch.int32, "contexts", 2)
    _dev(negatives, torch.int32, "negatives", 2)
    B = targets.shape[0]
    N = contexts.shape[1]
    K = negatives.shape[1]
    if contexts.shape[0] != B or negatives.shape[0] != B:
        raise ValueError("targets, contexts and negatives disagree on B")
    V, ld = _matrix(M_in, "M_in")
    if _matrix(M_out, "M_out") != (V, ld):
        raise ValueError("M_in and M_out must have the same shape and stride")
    D = M_in.shape[1] if D is None else D
    if isinstance(alpha, torch.Tensor):
        _dev(alpha, torch.float32, "alpha", 1)
        a_ptr, a_s = _ptr(alpha), 0.0
    else:
        a_ptr, a_s = None, float(alpha)
    if workspace is None:
        if sorted:
            n = step_batch_sorted_workspace_bytes(B, N, K, V, ld)
            if n == 0:
                raise W2VError(EINVAL if min(B, N, K) < 0 else EHIP,
                               "no workspace size for this batch (invalid shape "
                               "or failed sort size query)")
            workspace = torch.empty(n, dtype=torch.uint8, device=M_in.device)
        else:
            workspace = alloc_workspace(V, ld, M_in.device)
    if stats is not None:
        _dev(stats, torch.int64, "stats", 1)
        if stats.numel() < 5:
            raise ValueError("stats must have 5 entries (see w2v_train_epoch)")
    entry = lib().w2v_step_batch_sorted if sorted else lib().w2v_step_batch
    _check(entry(
        B, N, K, _ptr(targets), _ptr(contexts), _ptr(negatives), a_ptr, a_s,
        _ptr(M_in), _ptr(M_out), V, D, ld, _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(stats),
        _stream(stream)))
    return workspace


def build_vocab(raw, V_raw: int, min_count: int = 0, remap: bool = True,
                stream=None):
    """Counts, frequency ranks and min-count cut of a raw id stream on the GPU
    (w2v_build_vocab). Returns a dict of device tensors: ranked_counts
    int64[V_raw], rank_of int32[V_raw], corpus int32[T] (or None) and V (an
    int: this reads one value back from the device)."""
    import torch
    _dev(raw, torch.int32, "raw", 1)
    dev = raw.device
    T = raw.numel()
    ranked = torch.empty(V_raw, dtype=torch.int64, device=dev)
    rank_of = torch.empty(V_raw, dtype=torch.int32, device=dev)
    v_kept = torch.empty(1, dtype=torch.int32, device=dev)
    corpus = torch.empty(T, dtype=torch.int32, device=dev) if remap else None
    ws = torch.empty(int(lib().w2v_build_vocab_workspace_bytes(V_raw, T)),
                     dtype=torch.uint8, device=dev)
    _check(lib().w2v_build_vocab(_ptr(raw), T, V_raw, int(min_count), _ptr(ranked),
                                 _ptr(rank_of), _ptr(v_kept), _ptr(corpus), _ptr(ws),
                                 ws.numel(), _stream(stream)))
    return dict(ranked_counts=ranked, rank_of=rank_of, corpus=corpus,
                V=int(v_kept.item()))
