"""Writes planted_oracle_score.json: the CPU oracle's sequential 5-epoch run
on the planted-topic configuration (tests/planted.py) and its nearest-
neighbour topic score. Calls only the oracle and the seeded input
generators; takes about four hours on one core.

    python tests/golden/make_planted_score.py
"""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))
sys.path.insert(0, os.path.dirname(HERE))

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import planted  # noqa: E402


CONFIG = {"V": planted.V, "T": planted.T, "topics": planted.N_TOPICS,
          "D": planted.D, "window": planted.WINDOW, "K": planted.K,
          "sample": planted.SAMPLE, "epochs": planted.EPOCHS,
          "alpha0": planted.ALPHA0, "sentence_len": planted.SENTENCE,
          "corpus_seed": planted.CORPUS_SEED, "init_seed": planted.INIT_SEED,
          "sampling_seed": planted.SAMPLING_SEED, "table_size": planted.TABLE_SIZE,
          "checkpoints": list(planted.CHECKPOINTS)}


def write(epochs, checkpoints, complete):
    """Rewrites the JSON after every score, so a partial run keeps what it
    has measured ("complete" is set after the last epoch)."""
    out = {"complete": complete, "score": epochs[-1]["score"] if complete else None,
           "epochs": epochs, "checkpoints": checkpoints, "config": CONFIG,
           "source": "oracle.train_epoch, sequential, fp64 arithmetic, fp32 storage"}
    tmp = os.path.join(HERE, "planted_oracle_score.json.tmp")
    with open(tmp, "w") as f:
        json.dump(out, f, indent=1)
    os.replace(tmp, os.path.join(HERE, "planted_oracle_score.json"))


def main():
    t0 = time.time()
    corpus = planted.corpus()
    counts = np.bincount(corpus, minlength=planted.V).astype(np.int64)
    table, thr = oracle.build_tables(counts, 0.75, planted.SAMPLE, planted.TABLE_SIZE)
    M_in = planted.init_in()
    M_out = np.zeros_like(M_in)
    epochs, checkpoints = [], []
    for e in range(planted.EPOCHS):
        cuts = list(planted.CHECKPOINTS) if e == 0 else []
        bounds = [0] + cuts + [planted.T]
        n_e, l_e, c_e = 0, 0.0, 0.0
        for lo, hi in zip(bounds[:-1], bounds[1:]):
            s = oracle.Sampling(corpus, table, thr, window=planted.WINDOW, K=planted.K,
                                sentence_len=planted.SENTENCE, seed=planted.SAMPLING_SEED,
                                alpha0=planted.ALPHA0, epoch=e, n_epochs=planted.EPOCHS,
                                pos_begin=lo, pos_end=hi)
            n, b = oracle.train_epoch(s, M_in, M_out, n_buckets=1)
            n_e += int(n)
            l_e += float(b[0, 0])
            c_e += float(b[0, 1])
            if hi in cuts:
                checkpoints.append({"epoch": e, "tokens": hi,
                                    "score": planted.nn_topic_score(M_in)})
                print(json.dumps(checkpoints[-1]), flush=True)
                write(epochs, checkpoints, False)
        epochs.append({"epoch": e, "minibatches": n_e, "mean_loss_per_input": l_e / c_e,
                       "score": planted.nn_topic_score(M_in),
                       "elapsed_s": round(time.time() - t0, 1)})
        print(json.dumps(epochs[-1]), flush=True)
        write(epochs, checkpoints, e == planted.EPOCHS - 1)


if __name__ == "__main__":
    main()
