"""Writes largevocab_oracle.json: the CPU oracle's sequential epoch over the
large-vocabulary prefix (tests/largevocab.py): training loss per input word
and the held-out loss of the trained model. Calls only the oracle and the
seeded input generators; about two minutes on one core.

    python tests/golden/make_largevocab_trajectory.py
"""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))
sys.path.insert(0, os.path.dirname(HERE))

import numpy as np  # noqa: E402

import largevocab as lv  # noqa: E402
import oracle  # noqa: E402


def main():
    t0 = time.time()
    corpus = lv.corpus()
    table, thr = oracle.build_tables(lv.counts(), 0.75, lv.SAMPLE, 10**8)
    M_in = lv.init_in()
    M_out = np.zeros_like(M_in)
    s = oracle.Sampling(corpus, table, thr, window=lv.WINDOW, K=lv.K, seed=lv.SEED)
    n, b = oracle.train_epoch(s, M_in, M_out, n_buckets=1)
    held = lv.heldout_loss(M_in, M_out, *lv.heldout_ids(table))
    out = {"minibatches": int(n), "mean_loss_per_input": float(b[0, 0] / b[0, 1]),
           "inputs": float(b[0, 1]), "heldout_loss": held,
           "heldout_loss_initial": lv.heldout_loss(lv.init_in(), np.zeros_like(M_in),
                                                   *lv.heldout_ids(table)),
           "elapsed_s": round(time.time() - t0, 1),
           "source": "oracle.train_epoch, sequential, fp64 arithmetic, fp32 storage"}
    with open(os.path.join(HERE, "largevocab_oracle.json"), "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
