"""Planted-topic configuration and its score (shared by the GPU test and the
script that stores the oracle's score).

Corpus (reading R17): V = 71,290 words in 100 topics of 712-713 consecutive
ids, 17,000,000 tokens from a Markov chain that switches topic with
probability 0.05 per token, Zipf(1.0) inside a topic; D = 200, window 8,
K = 25, subsampling t = 1e-4, alpha 0.025 decaying linearly over 5 epochs.

Score: the fraction of all V words whose nearest neighbour by cosine
similarity of M_in rows (itself excluded) lies in the same topic (chance is
about 1%).
"""
import numpy as np

from paper_1611_06172_amd import configs, inputs

CFG = configs.Planted()
V = CFG.V
T = CFG.T
N_TOPICS = CFG.n_topics
D = CFG.D
WINDOW = CFG.window
K = CFG.K
SAMPLE = CFG.sample
EPOCHS = CFG.epochs
ALPHA0 = CFG.alpha0
SENTENCE = CFG.sentence
CORPUS_SEED = CFG.corpus_seed
INIT_SEED = CFG.init_seed
SAMPLING_SEED = CFG.sampling_seed
TABLE_SIZE = CFG.table_size
# Sentence-aligned token counts inside epoch 0 at which the score is also
# taken (the score saturates later in the run).
CHECKPOINTS = (100_000, 300_000, 1_000_000)


def corpus(T_=T):
    return inputs.planted_topic_corpus(T_, V, N_TOPICS, CFG.topic_zipf_s, CFG.switch,
                                       CORPUS_SEED)


def init_in():
    return inputs.init_matrix(V, D, "uniform", INIT_SEED)


def nn_topic_score(M_in, topics=None, chunk=4096):
    """Fraction of rows whose cosine nearest neighbour (not itself) shares
    the row's topic; fp64 on the CPU."""
    X = np.asarray(M_in, dtype=np.float64)
    X = X / np.maximum(np.linalg.norm(X, axis=1, keepdims=True), 1e-300)
    if topics is None:
        topics = inputs.topic_of(X.shape[0], N_TOPICS)
    hits = 0
    for a in range(0, X.shape[0], chunk):
        b = min(a + chunk, X.shape[0])
        S = X[a:b] @ X.T
        S[np.arange(b - a), np.arange(a, b)] = -np.inf
        nn = np.argmax(S, axis=1)
        hits += int((topics[nn] == topics[a:b]).sum())
    return hits / X.shape[0]
