"""The workloads the library is tested and measured on, one frozen dataclass
each, with a JSON round trip. They carry the shapes, hyper-parameters and
seeds; the generators that turn a seed into ids or matrices are in inputs.py.
The C ABI takes explicit scalar arguments, so these are only a convenient
record for the benchmark, the tests and the scripts that store expected
values.

Hyper-parameters follow the paper's Sec. 2 where it states them (dim 300,
negative 5, window 5, sample 1e-4, alpha 0.025); the corpora are synthetic
stand-ins for its one-billion-word benchmark.
"""
import dataclasses
import json
from typing import Tuple


@dataclasses.dataclass(frozen=True)
class Tiny:
    """200,000 i.i.d. Zipf(1.0) tokens over 1,000 words, D = 64, one epoch,
    no subsampling; M_in ~ U(-0.5/D, 0.5/D), M_out = 0."""
    T: int = 200_000
    V: int = 1_000
    zipf_s: float = 1.0
    D: int = 64
    window: int = 5
    K: int = 5
    sample: float = 0.0
    alpha0: float = 0.025
    epochs: int = 1
    corpus_seed: int = 1
    init_seed: int = 2


@dataclasses.dataclass(frozen=True)
class KernelTest:
    """One snapshot batch: B minibatches of 1 target, N inputs and K
    negatives, all i.i.d. Zipf(1.0) over V; M_in, M_out ~ N(0, 0.1^2)."""
    B: int = 65_536
    N: int = 10
    K: int = 5
    V: int = 100_000
    zipf_s: float = 1.0
    D: int = 300
    alpha: float = 0.025
    ids_seed: int = 3
    init_seed: int = 4


@dataclasses.dataclass(frozen=True)
class Planted:
    """Planted topics: a Markov chain over n_topics topics of consecutive
    ids, switching with probability `switch` per token, Zipf(1.0) inside a
    topic; scored by nearest-neighbour topic recovery."""
    V: int = 71_290
    T: int = 17_000_000
    n_topics: int = 100
    topic_zipf_s: float = 1.0
    switch: float = 0.05
    D: int = 200
    window: int = 8
    K: int = 25
    sample: float = 1e-4
    epochs: int = 5
    alpha0: float = 0.025
    sentence: int = 1000
    corpus_seed: int = 5
    init_seed: int = 2
    sampling_seed: int = 17
    table_size: int = 10**8


@dataclasses.dataclass(frozen=True)
class LargeVocab:
    """The throughput workload: 10^9 i.i.d. Zipf(1.07) tokens over 10^6
    words (inputs.zipf_corpus_hashed, the same ids on host and GPU), D = 300,
    window 5, K = 5, t = 1e-4."""
    T: int = 10**9
    V: int = 1_000_000
    zipf_s: float = 1.07
    D: int = 300
    window: int = 5
    K: int = 5
    sample: float = 1e-4
    alpha0: float = 0.025
    sentence: int = 1000
    corpus_seed: int = 6
    init_seed: int = 2
    sampling_seed: int = 1234
    table_size: int = 10**8


@dataclasses.dataclass(frozen=True)
class Sweep:
    """The shape sweep: the first T tokens of the throughput corpus at every
    D x K pair."""
    T: int = 10**8
    V: int = 1_000_000
    zipf_s: float = 1.07
    dims: Tuple[int, ...] = (100, 300, 600)
    negatives: Tuple[int, ...] = (5, 15, 64)
    window: int = 5
    sample: float = 1e-4
    corpus_seed: int = 6
    sampling_seed: int = 1234


ALL = {"tiny": Tiny, "kernel_test": KernelTest, "planted": Planted,
       "large_vocab": LargeVocab, "sweep": Sweep}


def to_json(cfg) -> str:
    """JSON of a config, with its kind."""
    name = next(k for k, c in ALL.items() if isinstance(cfg, c))
    return json.dumps({"kind": name, **dataclasses.asdict(cfg)}, sort_keys=True)


def from_json(text: str):
    """The config a to_json string describes (unknown fields are errors)."""
    d = json.loads(text)
    cls = ALL[d.pop("kind")]
    types = {f.name: f.type for f in dataclasses.fields(cls)}
    for k, v in d.items():
        if k not in types:
            raise ValueError(f"{cls.__name__} has no field {k!r}")
        if isinstance(v, list):
            d[k] = tuple(v)
    return cls(**d)
