/*
 * Plain CPU oracle for the HogBatch skip-gram negative-sampling (SGNS) SGD
 * step of Ji, Satish, Li and Dubey, "Parallelizing Word2Vec in Multi-Core and
 * Many-Core Architectures" (arXiv 1611.06172).
 *
 * TEST INFRASTRUCTURE ONLY. This code is the slow, single-threaded, fp64
 * reference that the GPU library is checked against. Only the tests, the
 * smoke check and the benchmark's CPU-baseline leg may load it. It shares no
 * source, header, table or constant with the GPU library: every function here
 * is written from the paper and from the published definitions it names.
 *
 * Conventions of this oracle (the readings of the paper it takes are listed
 * beside each function):
 *   - M_in and M_out are V x D fp32 matrices, row-major with leading dimension
 *     ld >= D (Sec. 1: one row of D floating point numbers per word).
 *   - All minibatch arithmetic is done in fp64 and rounded to fp32 once per
 *     element when written back.
 *   - Status: 0 on success, negative on invalid arguments.
 */
#ifndef W2V_ORACLE_H
#define W2V_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Philox4x64-10 block function (Salmon, Moraes, Dror, Shaw, "Parallel random
 * numbers: as easy as 1, 2, 3", SC'11). ctr[4], key[2] -> out[4]. */
void oracle_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2],
                          uint64_t out[4]);

/* 32-bit word `word` of the random stream attached to raw corpus position p in
 * epoch e: block j = word / 8 of Philox4x64-10 with counter (p, e, j, 0) and
 * key (seed, 0); the four 64-bit outputs are split low half first. */
uint32_t oracle_draw_u32(uint64_t seed, uint64_t p, uint64_t e, uint32_t word);

/* Sampling tables built from unigram counts (Sec. 2 hyper-parameters:
 * negative samples from the unigram distribution, sample = 1e-4).
 * neg_table[table_size]: word w owns the slots [bound(w-1), bound(w)) where
 *   bound(w) = floor(S_w / S_{V-1} * table_size), S_w = sum_{v<=w} c_v^power.
 * keep_thresh[V]: a position holding w is kept iff its draw r <= thresh[w];
 *   p_keep = sqrt(t/f) + t/f with f = c_w / sum(c); thresh = 0xFFFFFFFF when
 *   p_keep >= 1 or t == 0, else floor(p_keep * 2^32) - 1 (clamped at 0).
 * Either output may be NULL to skip it. */
int oracle_build_tables(const int64_t* counts, int32_t V, double neg_power,
                        double sample_t, int32_t* neg_table, int64_t table_size,
                        uint32_t* keep_thresh);

/* The sampling configuration shared by epoch training and minibatch export. */
typedef struct {
  const int32_t* corpus;      /* word ids x[0..T) */
  int64_t T;                  /* corpus length (the whole epoch) */
  int64_t pos_begin, pos_end; /* sentence-aligned sub-range [begin, end) */
  int32_t sentence_len;       /* raw tokens per sentence (last may be short) */
  int32_t window;             /* w: maximal half-width of the context window */
  int32_t K;                  /* negatives shared by one target's minibatch */
  const int32_t* neg_table;   /* [table_size] */
  int64_t table_size;
  const uint32_t* keep_thresh;/* [V] or NULL (no subsampling) */
  float alpha0;               /* starting learning rate */
  float min_alpha_frac;       /* floor of the linear decay, as a fraction */
  int32_t epoch, n_epochs;
  uint64_t seed;
} oracle_sampling;

/* Enumerates the minibatches of [pos_begin, pos_end) in processing order.
 * Minibatch m: target word out_targets[m] (row of M_out), its input context
 * words out_ctx[m*2w .. m*2w+2w) (rows of M_in, padded with -1), K negatives
 * out_negs[m*K ..] with out_mask[m*K ..] = 1 where the negative equals the
 * target, learning rate out_alpha[m] and raw corpus position out_pos[m].
 * Returns the number of minibatches; when it exceeds cap only the first cap
 * are written. Any output pointer may be NULL. Returns < 0 on bad arguments. */
int64_t oracle_minibatches(const oracle_sampling* s, int32_t* out_targets,
                           int32_t* out_ctx, int32_t* out_negs,
                           uint8_t* out_mask, float* out_alpha,
                           int64_t* out_pos, int64_t cap);

/* One HogBatch minibatch in fp64 (Sec. 1.1, Fig. 1 right; error term and
 * update directions of Alg. 1):
 *   X  = A O^T                  (N x (K+1)), A = context rows, O = [target; negatives]
 *   E  = alpha (l - sigma(X))   l = (1, 0, ..., 0); masked columns of E are 0
 *   dA = E O                    (N x D), update of the context rows of M_in
 *   dO = E^T A                  ((K+1) x D), update of the output rows of M_out
 * mask has K entries (column k+1 of E is zeroed when mask[k] != 0).
 * loss (may be NULL) receives sum_i [-log sigma(X_i0) - sum_{k unmasked}
 * log sigma(-X_i,k+1)]. X, dA, dO may be NULL. */
void oracle_sgns_delta(int32_t N, int32_t K, int32_t D, const double* A,
                       const double* O, const uint8_t* mask, double alpha,
                       double* X, double* dA, double* dO, double* loss);

/* oracle_sgns_delta plus the rounding-error scale of each update element:
 * sA[i][j] = sum_k |E_ik| |O_kj| and sO[k][j] = sum_i |E_ik| |A_ij| (the sums
 * of absolute products whose fp32 evaluation the GPU performs). sA, sO may be
 * NULL. */
void oracle_sgns_delta_scaled(int32_t N, int32_t K, int32_t D, const double* A,
                              const double* O, const uint8_t* mask,
                              double alpha, double* X, double* dA, double* dO,
                              double* loss, double* sA, double* sO);

/* Applies one minibatch to fp32 matrices in place: the gradients are computed
 * from the current (pre-update) rows, summed per destination row in fp64 and
 * rounded to fp32 once per element. ctx has N entries (-1 = absent). */
int oracle_apply_minibatch(float* M_in, float* M_out, int32_t V, int32_t D,
                           int32_t ld, int32_t N, const int32_t* ctx,
                           int32_t target, int32_t K, const int32_t* negs,
                           const uint8_t* mask, float alpha, double* loss,
                           int32_t* n_ctx);

/* A batch of B independent minibatches computed from one snapshot of the
 * input matrices, all updates summed in fp64 and rounded once at the end.
 * contexts [B][N] (-1 = absent), negatives [B][K]; a negative equal to its
 * target is masked. alpha is [B] or NULL (then alpha_scalar for all).
 * If S_in / S_out (V x D doubles, row stride D) are non-NULL they receive,
 * per element, |M0| plus, over every occurrence of the row in the batch, the
 * sum of absolute products forming that occurrence's update (sA / sO of
 * oracle_sgns_delta_scaled): the scale of the rounding error of evaluating
 * the update in fp32. */
int oracle_step_batch(int32_t B, int32_t N, int32_t K, const int32_t* targets,
                      const int32_t* contexts, const int32_t* negatives,
                      const float* alpha, float alpha_scalar, float* M_in,
                      float* M_out, int32_t V, int32_t D, int32_t ld,
                      double* S_in, double* S_out);

/* Sequential epoch over [pos_begin, pos_end): minibatches in processing order,
 * each applied before the next is formed. loss_buckets (may be NULL) holds
 * 2 * n_buckets doubles: [2b] += minibatch loss, [2b+1] += its number of
 * contexts, bucket b = floor(p * n_buckets / T) for the target position p.
 * Returns the number of minibatches applied, < 0 on bad arguments. */
int64_t oracle_train_epoch(const oracle_sampling* s, float* M_in, float* M_out,
                           int32_t V, int32_t D, int32_t ld,
                           double* loss_buckets, int32_t n_buckets);

/* Algorithm 1 (per-pair Hogwild SGD, one thread), sequential over the same
 * minibatches as oracle_train_epoch (targets, input words in window order,
 * learning rates), each input word with K negatives of its own:
 * oracle_pair_negative(s, p, i, k) is negative k of input word i of the
 * target at raw position p (draw 2 + iK + k of its stream). Returns the
 * number of targets applied, < 0 on bad arguments or an id outside [0, V).
 * Loss buckets as in oracle_train_epoch (the pairs' losses at the moment of
 * each pair). */
int32_t oracle_pair_negative(const oracle_sampling* s, int64_t p, int32_t i,
                             int32_t k);
int64_t oracle_pairwise_train_epoch(const oracle_sampling* s, float* M_in,
                                    float* M_out, int32_t V, int32_t D,
                                    int32_t ld, double* loss_buckets,
                                    int32_t n_buckets);

/* HogBatch with the K negatives shared by the G consecutive targets of a
 * group (retained indices [q0, q0+G), q0 a multiple of G, within a
 * sentence): negatives drawn at the group's first retained position, every
 * member's step from the rows as they were before the group, all updates
 * summed per row and rounded once. G = 1 is oracle_train_epoch. Returns the
 * number of minibatches (members) applied. A group's loss goes to the bucket
 * of its first member. */
int64_t oracle_grouped_train_epoch(const oracle_sampling* s, int32_t G,
                                   float* M_in, float* M_out, int32_t V,
                                   int32_t D, int32_t ld, double* loss_buckets,
                                   int32_t n_buckets);

#ifdef __cplusplus
}
#endif
#endif
