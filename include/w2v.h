/*
 * libw2v: HogBatch skip-gram negative-sampling SGD on MI355X (gfx950).
 *
 * Implements the shared-memory hot path of Ji, Satish, Li and Dubey,
 * "Parallelizing Word2Vec in Multi-Core and Many-Core Architectures"
 * (arXiv 1611.06172): for every target word, one minibatch of N input
 * (context) words and K negatives shared by those N words (Sec. 1.1, negative
 * sample sharing), whose dot products form an N x (K+1) block computed as one
 * small matrix product; the sigmoid error of Alg. 1 and both gradient
 * products follow, and the model updates are written back Hogwild-style (no
 * locks, conflicts between concurrent minibatches tolerated; Sec. 1.1,
 * "HogBatch").
 *
 * Conventions for every entry point:
 *   - M_in and M_out are V x D fp32 matrices, row-major, row stride ld >= D
 *     (floats). Word w is row w (Alg. 1: M_in holds input-word vectors, M_out
 *     output-word vectors). Columns D..ld-1 are never read or written.
 *   - "device" pointers are GPU global memory of the current HIP device;
 *     "host" pointers are ordinary CPU memory. The caller owns every buffer;
 *     the library keeps no pointer after a call returns and allocates no
 *     device memory.
 *   - GPU entry points are asynchronous on `stream` (a hipStream_t; NULL is
 *     the null stream). Results are visible once the caller synchronises it.
 *   - Return value: W2V_OK (0) or a negative W2V_E* code; w2v_last_error()
 *     then describes the failure. Arguments are validated on the host before
 *     any HIP call; a call that fails validation launches nothing.
 *   - Ids read from device memory (corpus, tables, batches) are always checked
 *     on the device: a minibatch that would touch a row outside [0, V) is
 *     skipped (no memory outside the given buffers is ever accessed), counted
 *     in the optional stats output, and recorded in the device's error word.
 *     The first GPU call on that device that starts after the skipping kernel
 *     has finished returns W2V_EDEVICE_FLAG, clears the word and launches
 *     nothing; w2v_device_status waits for a stream and reports the same.
 *     In the corpus, -1 marks a word removed from the vocabulary
 *     (w2v_build_vocab) and is no error: the position is dropped before
 *     windows form.
 *
 * Readings of points the paper leaves open (sentence cut, window shrink,
 * subsampling rule, negative distribution, learning-rate decay, random
 * numbers) are stated beside each entry point.
 */
#ifndef W2V_H
#define W2V_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define W2V_OK 0
#define W2V_EINVAL (-1)      /* an argument is out of range or NULL */
#define W2V_EHIP (-2)        /* the HIP runtime reported an error */
#define W2V_ENOMEM (-3)      /* a host allocation failed */
#define W2V_EUNSUPPORTED (-4)/* valid arguments outside the compiled shapes */
#define W2V_EDEVICE_FLAG (-5)/* an earlier call skipped work for an id outside
                                [0, V); nothing was launched by this call */
#define W2V_ENONFINITE (-6)  /* a loss bucket holds NaN or Inf (w2v_check_loss) */

/* Shape limits of the compiled kernels. The HogBatch kernels keep all N
 * input rows of a minibatch in registers, so they compile D <= 640 for up to
 * 10 input words (window <= 5), D <= 320 for up to 16 (window <= 8) and
 * D <= 128 for up to 32 (window <= 16); other valid combinations return
 * W2V_EUNSUPPORTED. Algorithm 1 compiles D <= 640 at every window. */
#define W2V_MAX_DIM 640          /* D */
#define W2V_MAX_WINDOW 16        /* window: up to 2*window input words */
#define W2V_MAX_NEGATIVE 64      /* K */
#define W2V_MAX_SENTENCE 1024    /* sentence_len */
#define W2V_MAX_BATCH_INPUTS 32  /* N of w2v_step_batch */

/* Partial rows per split row of w2v_train_epoch (one per XCD of MI355X). */
#define W2V_SPLIT_PARTS 8

/* Bytes of the library's static device scratch array, the partial rows of
 * w2v_train_epoch_noalloc (one copy per device, held until the process
 * ends): 2 * split_rows * W2V_SPLIT_PARTS * ld * 4 bytes must fit, e.g.
 * 204 split rows at ld = 320. */
#define W2V_NOALLOC_SCRATCH_BYTES 4194304

/* The `algorithm` argument of w2v_train_epoch. */
#define W2V_ALGORITHM_HOGBATCH 0  /* Sec. 1.1: minibatch, shared negatives */
#define W2V_ALGORITHM_PAIRWISE 1  /* Alg. 1: per-pair SGD, private negatives */
#define W2V_ALGORITHM_HOGBATCH_IMMEDIATE 2 /* Sec. 1.1, no pending input rows */

/* Version of this ABI (major * 100 + minor). */
int w2v_version(void);

/* Message of the last failed call on this thread ("" if none). The pointer
 * stays valid until the next call on the same thread. */
const char* w2v_last_error(void);

/* Sets up the library's per-device state on the current HIP device: the
 * device's error word (pinned host memory mapped into the device, 256 bytes,
 * held until the process ends) and the device address of the library's
 * static scratch array. Every GPU entry point does this itself on its first
 * call on a device, except w2v_train_epoch_noalloc, which allocates nothing
 * and so needs w2v_init to have run on the device first. Safe to call
 * repeatedly and from several threads. */
int w2v_init(void);

/* Waits for `stream` (a hipStream_t; NULL is the null stream), then returns
 * W2V_EDEVICE_FLAG (and clears the error word) if a kernel of this library on
 * the current device skipped a minibatch for an id outside [0, V) since the
 * word was last reported, else W2V_OK. */
int w2v_device_status(void* stream);

/* Failure detection for training (not in the paper, which reports no loss):
 * waits for `stream`, reads the n_buckets (sum, count) pairs of
 * loss_buckets (device double[n_buckets][2], as w2v_train_epoch fills them)
 * and returns W2V_ENONFINITE, naming the first such bucket, if a sum or a
 * count is NaN or Inf; W2V_OK otherwise. A NaN or Inf that reaches a row of
 * M_in or M_out makes the loss of every later minibatch reading the row
 * non-finite, so its bucket flags it. Launches nothing; copies 16 n_buckets
 * bytes to the host. W2V_EINVAL for n_buckets < 0 or a NULL pointer with
 * n_buckets > 0. */
int w2v_check_loss(const double* loss_buckets, int32_t n_buckets, void* stream);

/*
 * Sampling tables from unigram counts (host only; no HIP call).
 * Paper: Sec. 2 trains with 5 negative samples and sample = 1e-4; Alg. 1
 * draws each negative "from V". Readings:
 *   neg_table (host out, int32[table_size], may be NULL): word w owns slots
 *     [bound(w-1), bound(w)), bound(-1) = 0, bound(V-1) = table_size and
 *     bound(w) = floor(S_w / S_{V-1} * table_size) with
 *     S_w = sum_{v <= w} counts[v]^neg_power, summed left to right in fp64
 *     (neg_power = 0.75 gives the unigram^0.75 distribution).
 *   keep_thresh (host out, uint32[V], may be NULL): with f = counts[w] /
 *     sum(counts) and p = sqrt(t/f) + t/f, a position holding w is kept iff
 *     its 32-bit draw r <= keep_thresh[w]; keep_thresh[w] = 0xFFFFFFFF when
 *     t == 0, counts[w] == 0 or p >= 1, else max(floor(p * 2^32) - 1, 0).
 * counts: host int64[V], all >= 0 with a positive sum. table_size in
 * [1, 2^32). sample_t >= 0.
 */
int w2v_build_tables(const int64_t* counts, int32_t V, double neg_power,
                     double sample_t, int32_t* neg_table, int64_t table_size,
                     uint32_t* keep_thresh);

/*
 * Update-path choice for w2v_train_epoch (host only; no HIP call): the
 * number H of leading ids that should receive atomic updates. With the
 * sampling of w2v_build_tables, one minibatch writes the M_out row of word w
 * with probability about p_out(w) = rho_w + K q_w (rho: share of w among
 * kept words, q: its negative-sampling share) and the M_in row with
 * probability about p_in(w) = (window + 1) rho_w. With `inflight` minibatches
 * in flight, (inflight - 1) max(p_in, p_out) is the expected number of other
 * minibatches writing the row while one holds it. H is one more than the
 * largest id whose expected count reaches `tol` (0 if none), so every row at
 * or above H is rarely written concurrently. counts as for w2v_build_tables;
 * ids are expected to be ranked by frequency. Returns H >= 0, or a negative
 * W2V_E* code.
 */
int32_t w2v_hot_rows(const int64_t* counts, int32_t V, double neg_power,
                     double sample_t, int32_t window, int32_t K,
                     int64_t inflight, double tol);

/* Number of sentences w2v_train_epoch processes concurrently when called with
 * max_inflight = 0 on the current device (one wavefront each), or a negative
 * W2V_E* code: the wavefronts the device holds at once for this shape,
 * capped at max(1, floor(V / (4 group (2 window + K + 1)))). The cap keeps
 * the rows that the concurrent minibatches hold (up to 2 window input rows
 * and K + 1 output rows each, group times that for a group) under a quarter
 * of the vocabulary, so that a small vocabulary is not trained mostly from
 * stale rows; Hogwild staleness is what separates the concurrent epoch from
 * the sequential one (Sec. 1.1). At V = 10^6, window 5, K = 5 the cap
 * (15,625) is above what the GPU holds. A second cap, 131072 / (K + 1)
 * (2016 at K = 64), bounds how many concurrent sentences update the rows of
 * the words most often drawn as negatives, each from the row as it was
 * before the others' updates: at K = 64, D = 100 and alpha 0.025 the epoch
 * over a Zipf(1.07) vocabulary of 10^6 words learned with up to 2048
 * sentences in flight and diverged (NaN) with 2560. */
int64_t w2v_default_inflight(int32_t V, int32_t D, int32_t window, int32_t K,
                             int32_t group);

/* LDS slots per wavefront in which w2v_train_epoch (W2V_ALGORITHM_HOGBATCH,
 * group 1) collects pending input-row updates for this shape on the current
 * device (0: none), or a negative W2V_E* code. */
int32_t w2v_pending_slots(int32_t D, int32_t window, int32_t K);

/*
 * One Hogwild epoch (or a sentence-aligned part of one) of HogBatch SGD,
 * updating M_in and M_out in place on the GPU.
 *
 * Minibatch formation (readings; every random decision is a pure function of
 * (seed, raw position p, epoch) through Philox4x64-10, Salmon et al. SC'11,
 * with counter (p, epoch, j, 0) and key (seed, 0); block j's four 64-bit
 * outputs give 32-bit words 8j..8j+7, low half first):
 *   - the corpus is cut into sentences of sentence_len raw tokens (the last
 *     may be shorter); windows never cross a sentence;
 *   - position p is kept iff keep_thresh == NULL or word 0 <= keep_thresh[x_p];
 *   - each kept word (retained index q in its sentence) is a target; with
 *     b = floor(word1 * window / 2^32) and h = window - b its input words are
 *     the kept words at retained indices q-h..q+h except q; a target with no
 *     input word forms no minibatch;
 *   - negative k (k < K) is neg_table[floor(word(2+k) * table_size / 2^32)];
 *     a negative equal to the target is masked (contributes nothing);
 *   - alpha = fp32(alpha0 * max(min_alpha_frac, 1 - (epoch*T + p) /
 *     (n_epochs*T))), evaluated in IEEE fp64.
 * Minibatch step (Sec. 1.1, Alg. 1 error and update directions): with A the
 * input-word rows of M_in and O = [target row; negative rows] of M_out,
 *   X = A O^T, E = alpha * (l - sigma(X)), l = (1, 0, ..., 0),
 *   M_in[input words] += E O, M_out[target, negatives] += E^T A,
 * all from the rows as read at the start of the minibatch (repeated words
 * of one minibatch are merged, so each row is read and written once per
 * minibatch). Minibatches of one sentence run in order on one wavefront; up
 * to max_inflight sentences run concurrently and their updates interleave
 * without locks (Hogwild). max_inflight = 1 processes every minibatch in
 * sequence; 0 picks min(w2v_default_inflight(V, D, window, K, group),
 * ceil(S / 8)) for the S sentences of the range, so that they run in at
 * least 8 rounds (with every sentence of a short range in flight at once,
 * each would start from the initial model).
 * Pending input rows (W2V_ALGORITHM_HOGBATCH with group 1): consecutive
 * targets share most input words, so a wavefront adds the updates of a cold
 * input row (id >= max(hot_rows, split_rows)) to one of
 * w2v_pending_slots() LDS slots instead of M_in, reads the row as (M_in row
 * + pending updates) while its word is in the window, and adds the slot to
 * M_in atomically when it releases the word: when the slot is needed for
 * another word, when 2 * window targets pass without the word, and at the
 * end of the sentence. Every update reaches M_in before the call returns.
 * With one sentence in flight this changes only the order of the fp32
 * additions; with several, another sentence sees these updates late (as
 * late as the word stays in this sentence's window) and never loses them.
 * Rows below max(hot_rows, split_rows), which other sentences write
 * constantly, take their updates at once: deferring those lets the
 * concurrent sentences' stale steps pile up on them.
 * W2V_ALGORITHM_HOGBATCH_IMMEDIATE applies every update at the end of its
 * minibatch.
 * algorithm = W2V_ALGORITHM_PAIRWISE runs Alg. 1 instead (the original
 * per-pair Hogwild SGD, the paper's baseline) over the same targets, input
 * words and learning rates: each input word i in window order runs K+1
 * logistic regressions against the target and K negatives of its own
 * (draws 2 + iK + k of the target's stream; a draw equal to the target is
 * skipped); each pair reads the M_out row as moved by the pairs before it,
 * that row moves right after its pair, and the M_in row of i moves once,
 * after its K+1 pairs. A target with any negative outside [0, V) is skipped
 * and counted in stats[3]. split_rows must be 0 with this algorithm.
 * group (HogBatch algorithms; 1 is the paper's method): G in {2, 4, 8} shares the
 * K negatives among G consecutive targets instead of one target's input
 * words (the sharing of Sec. 1.1 widened). The retained targets of a
 * sentence are cut at multiples of G; the members of a group (its targets
 * with input words) take the negatives drawn at the group's first retained
 * position (draws 2..K+1 of its stream); a negative equal to a member's own
 * target is masked for that member; all members' steps read the rows as
 * they were before the group and their updates to a row are summed; a
 * group's loss goes to the bucket of its first member. Needs 2 window G <=
 * 64, 2 window + G <= 32 and G + K <= 32; G + K output columns are compiled
 * up to 16 for D <= 384 and 10 for D <= 640, up to 32 for D <= 128.
 * Update path: a row with id < hot_rows receives fp32 atomic adds (no update
 * is lost under concurrency); a row with id >= hot_rows is written back as
 * (value read + update) by a store written through to device scope, so a
 * concurrent update of the same row by another sentence may be
 * overwritten, as in Hogwild. With ids
 * ranked by frequency (id 0 the most frequent word) hot_rows selects the
 * frequent words, whose rows see concurrent updates; hot_rows >= V makes
 * every update atomic.
 * Split rows: atomics are performed at the memory side and those to one
 * address queue behind each other, so the few rows that nearly every
 * concurrent sentence writes (the head of the Zipf law) would stall the
 * whole memory system. A row with id < split_rows (regardless of hot_rows)
 * is therefore spread over W2V_SPLIT_PARTS partial rows in `workspace`:
 * each sentence adds its updates atomically to the partial row of its
 * wavefront's group, every read of the row returns the matrix row plus all
 * of its partial rows (so no update is hidden from any reader, as with a
 * single atomic row), and after the epoch the partial rows are added into
 * M_in/M_out and cleared. split_rows = 0 disables this; workspace may then
 * be NULL.
 *
 * corpus: device int32[T]. [pos_begin, pos_end) must start on a sentence
 * boundary and end on one or at T. M_in, M_out: device, see conventions.
 * neg_table: device int32[table_size]. keep_thresh: device uint32[V] or NULL.
 * loss_buckets: device double[2 * n_buckets] or NULL; for a minibatch of
 * target position p, bucket b = floor(p * n_buckets / T) receives
 * [2b] += sum_i [-log sigma(X_i0) - sum_{k unmasked} log sigma(-X_ik)] and
 * [2b+1] += N. workspace: device memory of at least
 * w2v_train_epoch_workspace_bytes(split_rows, ld) bytes, 256-byte aligned,
 * caller-owned, its
 * contents need not be initialised (the call clears what it uses), and it
 * must not be shared by calls that overlap in time. stats: device int64[5]
 * or NULL, accumulated into:
 * [0] minibatches applied, [1] sum of N over them, [2] raw positions
 * visited, [3] minibatches skipped for an id outside [0, V) (for the corpus:
 * positions holding such an id, -1 excepted), [4] rows read and written
 * back: per minibatch its distinct input and output rows, per group of
 * targets (group > 1) the distinct rows of the group, per input word of
 * Alg. 1 its row and K + 1 output rows.
 * Limits: 1 <= D <= W2V_MAX_DIM, 1 <= window <= W2V_MAX_WINDOW,
 * 0 <= K <= W2V_MAX_NEGATIVE, 1 <= sentence_len <= W2V_MAX_SENTENCE.
 */
int w2v_train_epoch(const int32_t* corpus, int64_t T, int64_t pos_begin,
                    int64_t pos_end, int32_t sentence_len, float* M_in,
                    float* M_out, int32_t V, int32_t D, int32_t ld,
                    int32_t window, int32_t K, const int32_t* neg_table,
                    int64_t table_size, const uint32_t* keep_thresh,
                    float alpha0, float min_alpha_frac, int32_t epoch,
                    int32_t n_epochs, uint64_t seed, double* loss_buckets,
                    int32_t n_buckets, int64_t* stats, int32_t max_inflight,
                    int32_t hot_rows, int32_t split_rows, void* workspace,
                    size_t workspace_bytes, int32_t algorithm, int32_t group,
                    void* stream);

/*
 * w2v_train_epoch for callers that cannot allocate (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * arguments, readings, limits and results, minus the workspace. The split
 * rows' partial rows live in the library's static device scratch array
 * (W2V_NOALLOC_SCRATCH_BYTES per device), so split_rows must satisfy
 * 2 * split_rows * W2V_SPLIT_PARTS * ld * 4 <= W2V_NOALLOC_SCRATCH_BYTES,
 * else W2V_EINVAL (nothing launched). The call allocates no device or
 * pinned memory and calls no hipMalloc or hipFree; w2v_init must have run
 * on the current device (else W2V_EINVAL). It clears the partial rows it
 * uses before the epoch (with a kernel, no memset) and after it. All calls
 * on one device share the one scratch array: calls that overlap in time on
 * the same device (other streams, other threads) race on it and must not
 * be issued. (A shape's launch configuration is computed on its first call
 * and cached in host memory.)
 */
int w2v_train_epoch_noalloc(const int32_t* corpus, int64_t T, int64_t pos_begin,
                            int64_t pos_end, int32_t sentence_len, float* M_in,
                            float* M_out, int32_t V, int32_t D, int32_t ld,
                            int32_t window, int32_t K, const int32_t* neg_table,
                            int64_t table_size, const uint32_t* keep_thresh,
                            float alpha0, float min_alpha_frac, int32_t epoch,
                            int32_t n_epochs, uint64_t seed, double* loss_buckets,
                            int32_t n_buckets, int64_t* stats, int32_t max_inflight,
                            int32_t hot_rows, int32_t split_rows, int32_t algorithm,
                            int32_t group, void* stream);

/* Workspace bytes w2v_train_epoch needs for split_rows rows of stride ld:
 * 2 * split_rows * W2V_SPLIT_PARTS * ld * 4 (0 when split_rows is 0). */
size_t w2v_train_epoch_workspace_bytes(int32_t split_rows, int32_t ld);

/*
 * Vocabulary of a raw id stream (GPU; the step before w2v_build_tables: the
 * paper's corpus is counted and its words ranked, Sec. 2). Counts every id
 * of raw[0..T) in [0, V_raw) (other values are not counted), ranks the ids
 * by count, descending, ties by increasing raw id, and keeps the words with
 * count >= max(min_count, 1).
 *   ranked_counts device int64[V_raw]: count of the word of rank r for
 *                 r < V, 0 after (the counts argument of w2v_build_tables);
 *   rank_of       device int32[V_raw]: the new id of raw id x (its rank), or
 *                 -1 when x is dropped;
 *   v_kept        device int32[1]: V, the number of words kept;
 *   corpus_out    device int32[T] or NULL: raw rewritten in new ids, -1 for
 *                 dropped words and ids outside [0, V_raw) (the epoch skips
 *                 such positions before forming windows).
 * With ids ranked this way id 0 is the most frequent word, as the update
 * tiers of w2v_train_epoch assume. workspace: device, 256-byte aligned,
 * >= w2v_build_vocab_workspace_bytes(V_raw, T) bytes, caller-owned; up to
 * V_raw = 4,194,304 the ids are counted by id range without atomics to
 * device memory, which takes about 4.3 T bytes of it (the stream reordered
 * by id range, and partial counts). The call is asynchronous on `stream`.
 */
size_t w2v_build_vocab_workspace_bytes(int32_t V_raw, int64_t T);
int w2v_build_vocab(const int32_t* raw, int64_t T, int32_t V_raw,
                    int64_t min_count, int64_t* ranked_counts,
                    int32_t* rank_of, int32_t* v_kept, int32_t* corpus_out,
                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * The minibatches w2v_train_epoch would form over [pos_begin, pos_end),
 * written out instead of applied (same arguments and readings as
 * w2v_train_epoch; the matrices are not needed): for every target word its
 * N input words and the K negatives they share (Sec. 1.1, negative sample
 * sharing; Alg. 1's problem statement: a target word, N input words, K
 * negatives drawn from V), with the sentence, window, subsampling, table and
 * learning-rate readings stated for w2v_train_epoch. This is the sampling
 * half of the epoch, exported so that it can be compared bit for bit with an
 * independent implementation. Outputs are indexed by raw
 * position r = p - pos_begin, P = pos_end - pos_begin:
 *   out_targets  device int32[P]: the target word, or -1 where position p
 *                forms no minibatch (not kept, or no input word);
 *   out_ctx      device int32[P][2*window]: input words in order, -1 padded;
 *   out_negs     device int32[P][K]; out_mask device uint8[P][K];
 *   out_alpha    device float[P].
 * Entries of out_ctx/out_negs/out_mask/out_alpha are written only where
 * out_targets != -1. stats as in w2v_train_epoch (may be NULL).
 */
int w2v_debug_minibatches(const int32_t* corpus, int64_t T, int64_t pos_begin,
                          int64_t pos_end, int32_t sentence_len, int32_t V,
                          int32_t window, int32_t K, const int32_t* neg_table,
                          int64_t table_size, const uint32_t* keep_thresh,
                          float alpha0, float min_alpha_frac, int32_t epoch,
                          int32_t n_epochs, uint64_t seed, int32_t* out_targets,
                          int32_t* out_ctx, int32_t* out_negs,
                          uint8_t* out_mask, float* out_alpha, int64_t* stats,
                          void* stream);

/* Bytes of workspace w2v_step_batch needs: two fp64 V x ld delta buffers. */
size_t w2v_step_batch_workspace_bytes(int32_t V, int32_t ld);

/*
 * One deterministic batch of B independent HogBatch minibatches against given
 * matrices. Each minibatch is the step of Sec. 1.1 for one target word, its
 * N input words and K shared negatives (Alg. 1's problem statement:
 * given M_in, M_out, alpha, a target word and N input words): X = A O^T,
 * E = alpha (l - sigma(X)), M_in[inputs] += E O, M_out[target, negatives]
 * += E^T A. Every gradient is computed from the matrices as they were on
 * entry: the paper computes a minibatch's products from the rows as read and
 * writes the updates back when its matrix product is done (Sec. 1.1); here
 * the whole batch shares that snapshot, so the result does not depend on the
 * order of the minibatches (a deterministic counterpart of the Hogwild
 * epoch, not a step the paper runs as such). The per-minibatch updates are
 * summed per element in fp64 (in `workspace`) and each touched element
 * becomes fp32(M + sum), one rounding per element. Elements whose summed
 * update is exactly 0 keep their bits.
 * targets: device int32[B]; contexts: device int32[B][N], -1 = absent;
 * negatives: device int32[B][K]; a negative equal to its target is masked.
 * alpha: device float[B], or NULL to use alpha_scalar for every minibatch.
 * workspace: device, >= w2v_step_batch_workspace_bytes(V, ld) bytes, 256-byte
 * aligned. stats: device int64[5] or NULL, as in w2v_train_epoch ([2] is
 * not used).
 * Limits: 0 <= N <= W2V_MAX_BATCH_INPUTS, 0 <= K <= W2V_MAX_NEGATIVE,
 * 1 <= D <= W2V_MAX_DIM.
 */
int w2v_step_batch(int32_t B, int32_t N, int32_t K, const int32_t* targets,
                   const int32_t* contexts, const int32_t* negatives,
                   const float* alpha, float alpha_scalar, float* M_in,
                   float* M_out, int32_t V, int32_t D, int32_t ld,
                   void* workspace, size_t workspace_bytes, int64_t* stats,
                   void* stream);

/* Bytes of workspace w2v_step_batch_sorted needs for B minibatches of N
 * input slots and K negatives over V rows of stride ld (0 on invalid
 * arguments or a failed query): staging rows for every update, sort keys
 * and values, per-chunk partial sums and the sort's temporaries. */
size_t w2v_step_batch_sorted_workspace_bytes(int32_t B, int32_t N, int32_t K,
                                             int32_t V, int32_t ld);

/*
 * The step of w2v_step_batch (same arguments, readings and limits) with
 * every row's updates summed in one fixed order: each minibatch's updates
 * are written to staging rows, sorted by row id with a stable radix sort
 * (so a row's updates stay in minibatch order) and summed per row in fp64
 * in that order, in chunks of 64 whose partial sums are added in chunk
 * order (grouped 32 chunks at a time). The result is the same bits on every run, and no atomics are
 * used. It may differ from w2v_step_batch, whose fp64 atomics add in
 * arrival order, in the last fp32 bit of an element.
 * Additional limit: B (N + K + 1) must fit in int32. workspace: device,
 * >= w2v_step_batch_sorted_workspace_bytes(B, N, K, V, ld) bytes, 256-byte
 * aligned, caller-owned, contents need not be initialised; calls that
 * overlap in time must not share it.
 */
int w2v_step_batch_sorted(int32_t B, int32_t N, int32_t K, const int32_t* targets,
                          const int32_t* contexts, const int32_t* negatives,
                          const float* alpha, float alpha_scalar, float* M_in,
                          float* M_out, int32_t V, int32_t D, int32_t ld,
                          void* workspace, size_t workspace_bytes, int64_t* stats,
                          void* stream);

#ifdef __cplusplus
}
#endif
#endif
