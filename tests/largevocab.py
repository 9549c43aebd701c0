"""The large-vocabulary workload on a prefix the oracle can follow (shared by
the GPU test and the script that stores the oracle's numbers): the first
1e8 tokens of the throughput benchmark's own corpus (i.i.d. Zipf(1.07) over
V = 1e6, inputs.zipf_corpus_hashed with the benchmark's seed, so the same ids
on the host and on the GPU), D = 300, K = 5, window 5, t = 1e-4, tables from
the prefix's counts, one epoch with the benchmark's sampling seed. The
held-out score is the mean SGNS loss per input word of 20,000 minibatches
drawn independently of the corpus."""
import numpy as np

from paper_1611_06172_amd import configs, inputs

CFG = configs.LargeVocab()
V, D, K, WINDOW, SAMPLE = CFG.V, CFG.D, CFG.K, CFG.window, CFG.sample
T = 100_000_000          # the prefix the oracle follows
CORPUS_SEED = CFG.corpus_seed
SEED = CFG.sampling_seed
N_BUCKETS = 10


def corpus(device="cpu"):
    """int32 torch tensor of the T tokens on `device`."""
    return inputs.zipf_corpus_hashed(T, V, CFG.zipf_s, CORPUS_SEED, device)


def counts(corpus_np):
    return inputs.word_counts(corpus_np, V)


def init_in():
    return inputs.init_matrix(V, D, "uniform", CFG.init_seed)


def heldout_ids(table):
    t = inputs.zipf_ids(20_000, V, 1.07, 77)
    c = inputs.zipf_ids((20_000, 6), V, 1.07, 78)
    n = table[np.random.default_rng(79).integers(0, len(table), (20_000, K))]
    return t, c, n


def heldout_loss(M_in, M_out, t, c, n):
    """Mean over minibatches and input words of -log sigma(a.o_t) -
    sum_k log sigma(-a.o_k) (negatives equal to the target skipped), fp64."""
    A = np.asarray(M_in, np.float64)[c]                      # [B, 6, D]
    O = np.asarray(M_out, np.float64)[np.concatenate([t[:, None], n], 1)]  # [B, K+1, D]
    X = np.matmul(A, np.ascontiguousarray(O.transpose(0, 2, 1)))
    sign = np.ones(K + 1)
    sign[1:] = -1
    L = np.logaddexp(0.0, -X * sign)                         # softplus(-sign x)
    mask = np.ones_like(L)
    mask[:, :, 1:] = (n != t[:, None])[:, None, :]
    return float((L * mask).sum() / (A.shape[0] * A.shape[1]))
