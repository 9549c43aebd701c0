"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle.

This module holds generators only (corpora, id batches, matrix initialisation,
word counts); it performs none of the method's arithmetic, and it is the one
piece of Python that both the GPU path's callers and the oracle's callers use.

Workload shapes follow the paper's training setup (Sec. 2: dim 300, 5
negatives, window 5, sample 1e-4, a vocabulary of about 1.1M words). The
one-billion-word corpus the paper trains on is not available here; i.i.d.
Zipfian streams with the same vocabulary size and hyper-parameters stand in for
it, and a planted-topic Markov stream stands in for the word-similarity
evaluation.
"""
from __future__ import annotations

import numpy as np


def zipf_pmf(V: int, s: float) -> np.ndarray:
    """Probabilities of word ids 0..V-1 proportional to (id + 1)^-s."""
    w = np.arange(1, V + 1, dtype=np.float64) ** (-float(s))
    return w / w.sum()


def zipf_cdf(V: int, s: float) -> np.ndarray:
    c = np.cumsum(zipf_pmf(V, s))
    c[-1] = 1.0
    return c


def zipf_ids(n, V: int, s: float, seed: int, chunk: int = 1 << 24) -> np.ndarray:
    """n i.i.d. Zipf(s) word ids over V words (inverse CDF, numpy PCG64).

    n may be an int or a shape tuple. Generated in chunks so that large corpora
    do not hold the uniforms in memory all at once.
    """
    shape = (n,) if np.ndim(n) == 0 else tuple(n)
    total = int(np.prod(shape))
    rng = np.random.Generator(np.random.PCG64(seed))
    cdf = zipf_cdf(V, s)
    out = np.empty(total, dtype=np.int32)
    for b in range(0, total, chunk):
        e = min(total, b + chunk)
        u = rng.random(e - b)
        out[b:e] = np.minimum(np.searchsorted(cdf, u, side="right"), V - 1)
    return out.reshape(shape)


def zipf_corpus_device(T: int, V: int, s: float, seed: int, device,
                       chunk: int = 1 << 27):
    """T i.i.d. Zipf(s) ids generated on a torch device (inverse CDF).

    Used for corpora too large to generate on the host in reasonable time; the
    ids are a seeded function of (seed, device type, torch version). Callers
    that need the same ids on the host copy them back.
    """
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    cdf = torch.from_numpy(zipf_cdf(V, s)).to(device)
    out = torch.empty(T, dtype=torch.int32, device=device)
    for b in range(0, T, chunk):
        e = min(T, b + chunk)
        u = torch.rand(e - b, generator=g, device=device, dtype=torch.float64)
        ids = torch.searchsorted(cdf, u, right=True)
        out[b:e] = torch.clamp(ids, max=V - 1).to(torch.int32)
    return out


_SPLITMIX_INC = 0x9E3779B97F4A7C15
_SPLITMIX_M1 = 0xBF58476D1CE4E5B9
_SPLITMIX_M2 = 0x94D049BB133111EB


def _i64(c: int) -> int:
    """A 64-bit constant as the signed value torch's int64 arithmetic uses."""
    return c - (1 << 64) if c >= (1 << 63) else c


def _splitmix64_torch(x):
    """SplitMix64 finaliser (Steele, Lea and Flood, OOPSLA 2014) of int64
    tensor x, in wrapping 64-bit arithmetic; logical right shifts are
    arithmetic shifts masked to the shifted width."""
    import torch

    def srl(z, k):
        return torch.bitwise_and(torch.bitwise_right_shift(z, k), (1 << (64 - k)) - 1)

    z = x + _i64(_SPLITMIX_INC)
    z = torch.bitwise_xor(z, srl(z, 30)) * _i64(_SPLITMIX_M1)
    z = torch.bitwise_xor(z, srl(z, 27)) * _i64(_SPLITMIX_M2)
    return torch.bitwise_xor(z, srl(z, 31))


def splitmix64_numpy(x: np.ndarray) -> np.ndarray:
    """The same finaliser on uint64 numpy arrays (numpy's uint64 arithmetic
    wraps modulo 2^64): the reference the torch version is tested against."""
    z = x.astype(np.uint64) + np.uint64(_SPLITMIX_INC)
    z = (z ^ (z >> np.uint64(30))) * np.uint64(_SPLITMIX_M1)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(_SPLITMIX_M2)
    return z ^ (z >> np.uint64(31))


def zipf_corpus_hashed(T: int, V: int, s: float, seed: int, device="cpu",
                       begin: int = 0, chunk: int = 1 << 26):
    """Tokens begin..begin+T-1 of an i.i.d. Zipf(s) stream over V words,
    the same ids on every torch device: token i takes u_i = top 53 bits of
    SplitMix64(seed * 2^40 + i) / 2^53 and the inverse CDF of the Zipf law
    (a binary search over fp64 cumulative probabilities, so integer and
    comparison work only). The throughput benchmark draws its 10^9-token
    corpus on the GPU and the oracle's stored results use the same ids,
    drawn on the host. Returns int32[T] on `device`."""
    import torch
    if not 0 <= seed < (1 << 22):
        raise ValueError("seed must be in [0, 2^22)")
    cdf = torch.from_numpy(zipf_cdf(V, s)).to(device)
    out = torch.empty(T, dtype=torch.int32, device=device)
    base = seed << 40
    for b in range(0, T, chunk):
        e = min(T, b + chunk)
        idx = torch.arange(base + begin + b, base + begin + e, dtype=torch.int64,
                           device=device)
        h = _splitmix64_torch(idx)
        top = torch.bitwise_and(torch.bitwise_right_shift(h, 11), (1 << 53) - 1)
        u = top.to(torch.float64) * (1.0 / (1 << 53))
        ids = torch.searchsorted(cdf, u, right=True)
        out[b:e] = torch.clamp(ids, max=V - 1).to(torch.int32)
    return out


def kernel_batch(B: int, N: int, K: int, V: int, s: float, seed: int):
    """Ids of B independent minibatches: targets [B], contexts [B, N],
    negatives [B, K], all i.i.d. Zipf(s) over V words."""
    ids = zipf_ids(B * (1 + N + K), V, s, seed).reshape(B, 1 + N + K)
    targets = np.ascontiguousarray(ids[:, 0])
    contexts = np.ascontiguousarray(ids[:, 1:1 + N])
    negatives = np.ascontiguousarray(ids[:, 1 + N:])
    return targets, contexts, negatives


def init_matrix(V: int, D: int, kind: str, seed: int, ld: int | None = None,
                scale: float | None = None) -> np.ndarray:
    """A V x ld fp32 matrix; columns >= D are zero.

    kind: "uniform" -> U(-0.5/D, 0.5/D) (scale overrides 0.5/D),
          "normal"  -> N(0, scale^2) (default scale 0.1),
          "zeros".
    """
    ld = D if ld is None else ld
    M = np.zeros((V, ld), dtype=np.float32)
    if kind == "zeros":
        return M
    rng = np.random.Generator(np.random.PCG64(seed))
    if kind == "uniform":
        a = 0.5 / D if scale is None else scale
        M[:, :D] = rng.uniform(-a, a, size=(V, D)).astype(np.float32)
    elif kind == "normal":
        sd = 0.1 if scale is None else scale
        M[:, :D] = rng.normal(0.0, sd, size=(V, D)).astype(np.float32)
    else:
        raise ValueError(kind)
    return M


def word_counts(corpus: np.ndarray, V: int) -> np.ndarray:
    """Occurrences of each word id in the corpus, int64[V]."""
    return np.bincount(np.asarray(corpus, dtype=np.int64), minlength=V).astype(np.int64)


def planted_topic_corpus(T: int, V: int, n_topics: int, s: float,
                         switch_p: float, seed: int) -> np.ndarray:
    """A Markov stream over n_topics latent topics.

    Topic k owns ids [floor(k V / n_topics), floor((k+1) V / n_topics)); within
    a topic, ids follow Zipf(s) over their offset + 1. The first topic is
    uniform; each token switches, with probability switch_p, to a topic drawn
    uniformly from the other n_topics - 1.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    bounds = (np.arange(n_topics + 1, dtype=np.int64) * V) // n_topics
    switch = rng.random(T) < switch_p
    switch[0] = False
    jumps = rng.integers(1, n_topics, size=T)
    topic = np.empty(T, dtype=np.int64)
    t0 = int(rng.integers(0, n_topics))
    # topic_t = (t0 + sum of jumps at switch points up to t) mod n_topics
    steps = np.where(switch, jumps, 0)
    topic[:] = (t0 + np.cumsum(steps)) % n_topics
    u = rng.random(T)
    out = np.empty(T, dtype=np.int32)
    for k in range(n_topics):
        sel = topic == k
        size = int(bounds[k + 1] - bounds[k])
        cdf = zipf_cdf(size, s)
        off = np.minimum(np.searchsorted(cdf, u[sel], side="right"), size - 1)
        out[sel] = (bounds[k] + off).astype(np.int32)
    return out


def topic_of(V: int, n_topics: int) -> np.ndarray:
    """Topic label of every word id for planted_topic_corpus."""
    bounds = (np.arange(n_topics + 1, dtype=np.int64) * V) // n_topics
    ids = np.arange(V, dtype=np.int64)
    return (np.searchsorted(bounds, ids, side="right") - 1).astype(np.int32)
