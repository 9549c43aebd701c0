"""Writes largevocab_oracle.json: the CPU oracle's sequential epoch over the
large-vocabulary prefix (tests/largevocab.py, the first 1e8 tokens of the
throughput benchmark's corpus), run as ten sentence-aligned ranges of 1e7
tokens (resume is bitwise, so this is one epoch): the training loss per
input word in ten buckets of raw position, and the held-out loss of the
model after each range. Calls only the oracle and the seeded input
generators; about half an hour on one core. The file is rewritten after
every range.

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
    corpus = lv.corpus().numpy()
    table, thr = oracle.build_tables(lv.counts(corpus), 0.75, lv.SAMPLE, 10**8)
    held_ids = lv.heldout_ids(table)
    M_in = lv.init_in()
    M_out = np.zeros_like(M_in)
    out = {"T": lv.T, "n_buckets": lv.N_BUCKETS,
           "heldout_loss_initial": lv.heldout_loss(M_in, M_out, *held_ids),
           "source": "oracle.train_epoch, sequential, fp64 arithmetic, fp32 storage; "
                     "tests/golden/make_largevocab_trajectory.py",
           "buckets": [], "heldout_after_range": [], "minibatches": 0}
    step = lv.T // lv.N_BUCKETS
    buckets = np.zeros((lv.N_BUCKETS, 2))
    for r in range(lv.N_BUCKETS):
        s = oracle.Sampling(corpus, table, thr, window=lv.WINDOW, K=lv.K, seed=lv.SEED,
                            pos_begin=r * step, pos_end=(r + 1) * step)
        n, b = oracle.train_epoch(s, M_in, M_out, n_buckets=lv.N_BUCKETS)
        buckets += b
        out["minibatches"] += int(n)
        out["buckets"] = buckets.tolist()
        out["heldout_after_range"].append(lv.heldout_loss(M_in, M_out, *held_ids))
        out["elapsed_s"] = round(time.time() - t0, 1)
        out["complete"] = r == lv.N_BUCKETS - 1
        with open(os.path.join(HERE, "largevocab_oracle.json"), "w") as f:
            json.dump(out, f, indent=1)
        print(f"range {r}: {n} minibatches, loss {b[r, 0] / b[r, 1]:.4f}, held-out "
              f"{out['heldout_after_range'][-1]:.4f}, {out['elapsed_s']} s", flush=True)


if __name__ == "__main__":
    main()
