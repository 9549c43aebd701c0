"""Checkpoint and resume of a training run.

Every random draw of an epoch is a function of (seed, epoch, raw position)
and the learning rate is a function of the raw position (the counter-based
sampling of w2v_train_epoch), so an epoch cut at sentence boundaries into
ranges [pos_begin, pos_end) and run range by range forms exactly the
minibatches of the uncut epoch. A checkpoint therefore needs only the two
matrices and a small record: seed, epoch, schedule length, the next raw
position to train (a sentence boundary), and a hash of everything else the
run depends on (hyper-parameters, tables, a fingerprint of the corpus).

Layout of a checkpoint directory:
    state.json              the record, written last and replaced atomically
    M_in.<g>.npy, M_out.<g>.npy, loss.<g>.npy (optional)
                            the arrays of generation g, which state.json names
A save writes the new generation's arrays, then replaces state.json, then
removes the older generations, so a run killed at any point leaves a
state.json that names complete arrays.
"""
import hashlib
import json
import os
from typing import Optional

import numpy as np

FORMAT = 1
STATE = "state.json"


def _host(a) -> np.ndarray:
    """A host numpy view or copy of a numpy array or torch tensor."""
    if isinstance(a, np.ndarray):
        return a
    return a.detach().cpu().numpy()


def corpus_fingerprint(corpus, n: int = 1 << 20) -> str:
    """SHA-256 over the corpus length and its first and last n ids: a cheap
    identity for a stream that may be billions of ids long."""
    T = int(corpus.shape[0])
    h = hashlib.sha256(str(T).encode())
    h.update(np.ascontiguousarray(_host(corpus[:n])).tobytes())
    h.update(np.ascontiguousarray(_host(corpus[max(0, T - n):])).tobytes())
    return h.hexdigest()


def config_hash(config: dict, *arrays) -> str:
    """SHA-256 of the config (as sorted JSON) and of each array's dtype, shape
    and bytes (None entries hash as absent)."""
    h = hashlib.sha256(json.dumps(config, sort_keys=True).encode())
    for a in arrays:
        if a is None:
            h.update(b"none")
            continue
        x = np.ascontiguousarray(_host(a))
        h.update(f"{x.dtype.str}{x.shape}".encode())
        h.update(x.tobytes())
    return h.hexdigest()


def save(path: str, M_in, M_out, state: dict, loss_buckets=None) -> dict:
    """Writes a checkpoint of the matrices (and loss buckets) with `state`
    (JSON-serialisable: seed, epoch, n_epochs, next_pos, config_hash, ...).
    Returns the record written."""
    os.makedirs(path, exist_ok=True)
    old = _read_state(path)
    gen = (old["generation"] + 1) if old else 0
    files = {"M_in": f"M_in.{gen}.npy", "M_out": f"M_out.{gen}.npy"}
    arrays = {"M_in": M_in, "M_out": M_out}
    if loss_buckets is not None:
        files["loss"] = f"loss.{gen}.npy"
        arrays["loss"] = loss_buckets
    for k, name in files.items():
        tmp = os.path.join(path, name + ".tmp")
        with open(tmp, "wb") as f:
            np.save(f, np.ascontiguousarray(_host(arrays[k])), allow_pickle=False)
            f.flush()
            os.fsync(f.fileno())
        os.replace(tmp, os.path.join(path, name))
    record = dict(state, format=FORMAT, generation=gen, files=files)
    tmp = os.path.join(path, STATE + ".tmp")
    with open(tmp, "w") as f:
        json.dump(record, f, indent=1, sort_keys=True)
        f.flush()
        os.fsync(f.fileno())
    os.replace(tmp, os.path.join(path, STATE))
    if old:
        for name in old["files"].values():
            if name not in files.values():
                try:
                    os.remove(os.path.join(path, name))
                except FileNotFoundError:
                    pass
    return record


def _read_state(path: str) -> Optional[dict]:
    p = os.path.join(path, STATE)
    if not os.path.exists(p):
        return None
    with open(p) as f:
        rec = json.load(f)
    if rec.get("format") != FORMAT:
        raise ValueError(f"{p}: unknown checkpoint format {rec.get('format')}")
    return rec


def load(path: str, expect_hash: Optional[str] = None):
    """Returns (record, arrays) of the checkpoint at `path`, or (None, None)
    if there is none; arrays maps "M_in", "M_out" (and "loss" if saved) to
    host numpy arrays. Raises ValueError if expect_hash is given and the
    checkpoint belongs to another configuration."""
    rec = _read_state(path)
    if rec is None:
        return None, None
    if expect_hash is not None and rec.get("config_hash") != expect_hash:
        raise ValueError(f"{path}: checkpoint of another configuration "
                         f"({rec.get('config_hash')} != {expect_hash})")
    arrays = {k: np.load(os.path.join(path, name), allow_pickle=False)
              for k, name in rec["files"].items()}
    return rec, arrays


def train_epoch_resumable(path: str, corpus, M_in, M_out, neg_table, keep_thresh=None,
                          *, epoch: int = 0, n_epochs: int = 1, seed: int = 0,
                          chunk_sentences: int = 1000, sentence_len: int = 1000,
                          loss_buckets=None, max_chunks: Optional[int] = None,
                          corpus_id: Optional[str] = None, **kw) -> dict:
    """One epoch of w2v.train_epoch run in ranges of chunk_sentences
    sentences, with a checkpoint at `path` after each range. If `path` holds
    a checkpoint of the same configuration and epoch, the matrices (and loss
    buckets) are restored into M_in / M_out (/ loss_buckets) and training
    continues from its next position; a checkpoint of a later epoch, or of
    this epoch completed, means there is nothing to do. max_chunks stops
    after that many ranges (a run cut short). Other keyword arguments go to
    w2v.train_epoch; the scalar ones, the tables and the corpus identity
    (corpus_id, else corpus_fingerprint) make up the configuration hash.
    Returns the last record."""
    import torch

    from . import w2v

    T = int(corpus.numel())
    V, ld = int(M_in.shape[0]), int(M_in.stride(0))
    # scalar arguments shape the run; tensors (stats, workspace) and the
    # stream do not
    scalars = {k: v for k, v in kw.items()
               if k != "stream" and (v is None or isinstance(v, (bool, int, float, str)))}
    config = dict(scalars, T=T, V=V, D=int(kw.get("D") or M_in.shape[1]), ld=ld,
                  n_epochs=n_epochs, seed=seed, sentence_len=sentence_len,
                  corpus=corpus_id or corpus_fingerprint(corpus),
                  loss_buckets=None if loss_buckets is None else list(loss_buckets.shape))
    h = config_hash(config, neg_table, keep_thresh)
    rec, arrays = load(path, expect_hash=h)
    pos = 0
    if rec is not None:
        if rec["epoch"] > epoch or (rec["epoch"] == epoch and rec["next_pos"] >= T):
            return rec
        if rec["epoch"] == epoch:
            pos = int(rec["next_pos"])
        elif rec["next_pos"] < T:
            raise ValueError(f"{path}: epoch {rec['epoch']} stopped at position "
                             f"{rec['next_pos']}; finish it before epoch {epoch}")
        # restore the matrices the record was taken with (the end of the
        # previous epoch, or the middle of this one)
        M_in.copy_(torch.from_numpy(arrays["M_in"]))
        M_out.copy_(torch.from_numpy(arrays["M_out"]))
        if loss_buckets is not None and "loss" in arrays and rec["epoch"] == epoch:
            loss_buckets.copy_(torch.from_numpy(arrays["loss"]))
    if pos % sentence_len != 0:
        raise ValueError(f"{path}: next position {pos} is not a sentence boundary")
    step = chunk_sentences * sentence_len
    done = 0
    while pos < T and (max_chunks is None or done < max_chunks):
        end = min(T, pos + step)
        w2v.train_epoch(corpus, M_in, M_out, neg_table, keep_thresh, epoch=epoch,
                        n_epochs=n_epochs, seed=seed, pos_begin=pos, pos_end=end,
                        sentence_len=sentence_len, loss_buckets=loss_buckets, **kw)
        torch.cuda.synchronize(M_in.device)
        pos = end
        done += 1
        rec = save(path, M_in, M_out,
                   dict(seed=seed, epoch=epoch, n_epochs=n_epochs, next_pos=pos,
                        config_hash=h, config=config),
                   loss_buckets=loss_buckets)
    return rec
