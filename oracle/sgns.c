/*
 * Oracle: the HogBatch SGNS minibatch step, a batch of snapshot steps and a
 * sequential epoch. TEST INFRASTRUCTURE ONLY.
 *
 * The minibatch of Sec. 1.1 (Fig. 1 right) batches, for one target word and
 * its N input words, the dot products of Alg. 1 into one matrix product, then
 * writes the model updates back at the end of that product. Per input word i
 * and output column k (column 0 = target, label 1; columns 1..K = negatives,
 * label 0) Alg. 1 fixes: inner product of the M_in row of i with the M_out row
 * of k, error = label - sigma(inner product), M_out row of k moves by
 * alpha * error * (M_in row of i), M_in row of i moves by alpha * sum_k error *
 * (M_out row of k). In the minibatch form all inner products use the rows as
 * they were before the minibatch (the updates are written back after the
 * product), so the step is
 *   X = A O^T,  E = alpha (l - sigma(X)),  dA = E O,  dO = E^T A.
 * These are alpha times the negative gradient of the skip-gram
 * negative-sampling loss  sum_i [ -log sigma(X_i0) - sum_k log sigma(-X_ik) ].
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include "oracle.h"
#include "oracle_internal.h"

/* Logistic function, evaluated without overflow for either sign. */
static double sigma(double x) {
  if (x >= 0.0) return 1.0 / (1.0 + exp(-x));
  double ex = exp(x);
  return ex / (1.0 + ex);
}

/* log(sigma(x)), evaluated without overflow for either sign. */
static double log_sigma(double x) {
  if (x >= 0.0) return -log1p(exp(-x));
  return x - log1p(exp(x));
}

void oracle_sgns_delta(int32_t N, int32_t K, int32_t D, const double* A,
                       const double* O, const uint8_t* mask, double alpha,
                       double* X, double* dA, double* dO, double* loss) {
  oracle_sgns_delta_scaled(N, K, D, A, O, mask, alpha, X, dA, dO, loss, NULL,
                           NULL);
}

void oracle_sgns_delta_scaled(int32_t N, int32_t K, int32_t D, const double* A,
                              const double* O, const uint8_t* mask,
                              double alpha, double* X, double* dA, double* dO,
                              double* loss, double* sA, double* sO) {
  const int32_t C = K + 1;
  double* x = (double*)malloc(sizeof(double) * (size_t)(N * C + 1));
  double* e = (double*)malloc(sizeof(double) * (size_t)(N * C + 1));
  double total_loss = 0.0;
  for (int32_t i = 0; i < N; ++i) {
    for (int32_t k = 0; k < C; ++k) {
      double inner = 0.0;
      for (int32_t j = 0; j < D; ++j) inner += A[(size_t)i * D + j] * O[(size_t)k * D + j];
      x[i * C + k] = inner;
      int masked = (k > 0 && mask != NULL && mask[k - 1] != 0);
      double label = (k == 0) ? 1.0 : 0.0;
      e[i * C + k] = masked ? 0.0 : alpha * (label - sigma(inner));
      if (!masked) total_loss -= (k == 0) ? log_sigma(inner) : log_sigma(-inner);
    }
  }
  if (X != NULL) memcpy(X, x, sizeof(double) * (size_t)(N * C));
  if (dA != NULL) {
    for (int32_t i = 0; i < N; ++i)
      for (int32_t j = 0; j < D; ++j) {
        double acc = 0.0;
        for (int32_t k = 0; k < C; ++k) acc += e[i * C + k] * O[(size_t)k * D + j];
        dA[(size_t)i * D + j] = acc;
      }
  }
  if (dO != NULL) {
    for (int32_t k = 0; k < C; ++k)
      for (int32_t j = 0; j < D; ++j) {
        double acc = 0.0;
        for (int32_t i = 0; i < N; ++i) acc += e[i * C + k] * A[(size_t)i * D + j];
        dO[(size_t)k * D + j] = acc;
      }
  }
  if (sA != NULL) {
    for (int32_t i = 0; i < N; ++i)
      for (int32_t j = 0; j < D; ++j) {
        double acc = 0.0;
        for (int32_t k = 0; k < C; ++k)
          acc += fabs(e[i * C + k]) * fabs(O[(size_t)k * D + j]);
        sA[(size_t)i * D + j] = acc;
      }
  }
  if (sO != NULL) {
    for (int32_t k = 0; k < C; ++k)
      for (int32_t j = 0; j < D; ++j) {
        double acc = 0.0;
        for (int32_t i = 0; i < N; ++i)
          acc += fabs(e[i * C + k]) * fabs(A[(size_t)i * D + j]);
        sO[(size_t)k * D + j] = acc;
      }
  }
  if (loss != NULL) *loss = total_loss;
  free(x);
  free(e);
}

/* Gathers the rows of the minibatch; returns the number of present input
 * words, or -1 when an id is out of range. rows_in/rows_out receive ids. */
static int32_t gather(const float* M_in, const float* M_out, int32_t V,
                      int32_t D, int32_t ld, int32_t N, const int32_t* ctx,
                      int32_t target, int32_t K, const int32_t* negs,
                      double* A, double* O, int32_t* rows_in,
                      int32_t* rows_out) {
  int32_t n = 0;
  for (int32_t i = 0; i < N; ++i) {
    if (ctx[i] < 0) continue;
    if (ctx[i] >= V) return -1;
    rows_in[n] = ctx[i];
    for (int32_t j = 0; j < D; ++j)
      A[(size_t)n * D + j] = (double)M_in[(size_t)ctx[i] * ld + j];
    ++n;
  }
  for (int32_t k = 0; k <= K; ++k) {
    int32_t id = (k == 0) ? target : negs[k - 1];
    if (id < 0 || id >= V) return -1;
    rows_out[k] = id;
    for (int32_t j = 0; j < D; ++j)
      O[(size_t)k * D + j] = (double)M_out[(size_t)id * ld + j];
  }
  return n;
}

/* Sums the update rows per destination id in fp64 and rounds once. */
static void write_back(float* M, int32_t D, int32_t ld, int32_t n_rows,
                       const int32_t* rows, const double* dM, double* acc) {
  for (int32_t r = 0; r < n_rows; ++r) {
    int first = 1;
    for (int32_t q = 0; q < r; ++q)
      if (rows[q] == rows[r]) first = 0;
    if (!first) continue;
    for (int32_t j = 0; j < D; ++j) acc[j] = 0.0;
    for (int32_t q = r; q < n_rows; ++q) {
      if (rows[q] != rows[r]) continue;
      for (int32_t j = 0; j < D; ++j) acc[j] += dM[(size_t)q * D + j];
    }
    float* row = M + (size_t)rows[r] * ld;
    for (int32_t j = 0; j < D; ++j) row[j] = (float)((double)row[j] + acc[j]);
  }
}

int oracle_apply_minibatch(float* M_in, float* M_out, int32_t V, int32_t D,
                           int32_t ld, int32_t N, const int32_t* ctx,
                           int32_t target, int32_t K, const int32_t* negs,
                           const uint8_t* mask, float alpha, double* loss,
                           int32_t* n_ctx) {
  if (M_in == NULL || M_out == NULL || V <= 0 || D <= 0 || ld < D || N < 0 ||
      K < 0 || (N > 0 && ctx == NULL) || (K > 0 && negs == NULL))
    return -1;
  const int32_t C = K + 1;
  double* A = (double*)malloc(sizeof(double) * (size_t)(N + 1) * D);
  double* O = (double*)malloc(sizeof(double) * (size_t)C * D);
  double* dA = (double*)malloc(sizeof(double) * (size_t)(N + 1) * D);
  double* dO = (double*)malloc(sizeof(double) * (size_t)C * D);
  double* acc = (double*)malloc(sizeof(double) * (size_t)D);
  int32_t* rows_in = (int32_t*)malloc(sizeof(int32_t) * (size_t)(N + 1));
  int32_t* rows_out = (int32_t*)malloc(sizeof(int32_t) * (size_t)C);
  int status = 0;
  int32_t n = gather(M_in, M_out, V, D, ld, N, ctx, target, K, negs, A, O,
                     rows_in, rows_out);
  if (n < 0) {
    status = -1;
  } else if (n > 0) {
    double l = 0.0;
    oracle_sgns_delta(n, K, D, A, O, mask, (double)alpha, NULL, dA, dO, &l);
    write_back(M_in, D, ld, n, rows_in, dA, acc);
    write_back(M_out, D, ld, C, rows_out, dO, acc);
    if (loss != NULL) *loss = l;
  } else if (loss != NULL) {
    *loss = 0.0;
  }
  if (n_ctx != NULL) *n_ctx = n < 0 ? 0 : n;
  free(A); free(O); free(dA); free(dO); free(acc); free(rows_in); free(rows_out);
  return status;
}

int oracle_step_batch(int32_t B, int32_t N, int32_t K, const int32_t* targets,
                      const int32_t* contexts, const int32_t* negatives,
                      const float* alpha, float alpha_scalar, float* M_in,
                      float* M_out, int32_t V, int32_t D, int32_t ld,
                      double* S_in, double* S_out) {
  if (B < 0 || N < 0 || K < 0 || V <= 0 || D <= 0 || ld < D ||
      M_in == NULL || M_out == NULL || (B > 0 && targets == NULL) ||
      (B > 0 && N > 0 && contexts == NULL) ||
      (B > 0 && K > 0 && negatives == NULL))
    return -1;
  const int32_t C = K + 1;
  const size_t VD = (size_t)V * (size_t)D;
  double* dM_in = (double*)calloc(VD, sizeof(double));
  double* dM_out = (double*)calloc(VD, sizeof(double));
  uint8_t* touched_in = (uint8_t*)calloc((size_t)V, 1);
  uint8_t* touched_out = (uint8_t*)calloc((size_t)V, 1);
  double* A = (double*)malloc(sizeof(double) * (size_t)(N + 1) * D);
  double* O = (double*)malloc(sizeof(double) * (size_t)C * D);
  double* dA = (double*)malloc(sizeof(double) * (size_t)(N + 1) * D);
  double* dO = (double*)malloc(sizeof(double) * (size_t)C * D);
  double* sA = (double*)malloc(sizeof(double) * (size_t)(N + 1) * D);
  double* sO = (double*)malloc(sizeof(double) * (size_t)C * D);
  int32_t* rows_in = (int32_t*)malloc(sizeof(int32_t) * (size_t)(N + 1));
  int32_t* rows_out = (int32_t*)malloc(sizeof(int32_t) * (size_t)C);
  uint8_t* mask = (uint8_t*)malloc((size_t)K + 1);
  int status = 0;
  if (!dM_in || !dM_out || !touched_in || !touched_out || !A || !O || !dA ||
      !dO || !sA || !sO || !rows_in || !rows_out || !mask) {
    status = -2;
    goto done;
  }
  if (S_in != NULL)
    for (int32_t r = 0; r < V; ++r)
      for (int32_t j = 0; j < D; ++j)
        S_in[(size_t)r * D + j] = fabs((double)M_in[(size_t)r * ld + j]);
  if (S_out != NULL)
    for (int32_t r = 0; r < V; ++r)
      for (int32_t j = 0; j < D; ++j)
        S_out[(size_t)r * D + j] = fabs((double)M_out[(size_t)r * ld + j]);
  /* Validate every id before any arithmetic. */
  for (int32_t b = 0; b < B; ++b) {
    if (targets[b] < 0 || targets[b] >= V) { status = -1; goto done; }
    for (int32_t i = 0; i < N; ++i) {
      int32_t id = contexts[(size_t)b * N + i];
      if (id < -1 || id >= V) { status = -1; goto done; }
    }
    for (int32_t k = 0; k < K; ++k) {
      int32_t id = negatives[(size_t)b * K + k];
      if (id < 0 || id >= V) { status = -1; goto done; }
    }
  }
  for (int32_t b = 0; b < B; ++b) {
    const int32_t* negs = negatives + (size_t)b * K;
    for (int32_t k = 0; k < K; ++k) mask[k] = (uint8_t)(negs[k] == targets[b]);
    int32_t n = gather(M_in, M_out, V, D, ld, N, contexts + (size_t)b * N,
                       targets[b], K, negs, A, O, rows_in, rows_out);
    if (n <= 0) continue;
    double a = alpha != NULL ? (double)alpha[b] : (double)alpha_scalar;
    oracle_sgns_delta_scaled(n, K, D, A, O, mask, a, NULL, dA, dO, NULL, sA,
                             sO);
    for (int32_t i = 0; i < n; ++i) {
      size_t base = (size_t)rows_in[i] * D;
      touched_in[rows_in[i]] = 1;
      for (int32_t j = 0; j < D; ++j) {
        dM_in[base + j] += dA[(size_t)i * D + j];
        if (S_in != NULL) S_in[base + j] += sA[(size_t)i * D + j];
      }
    }
    for (int32_t k = 0; k < C; ++k) {
      if (k > 0 && mask[k - 1]) continue; /* masked column: no update */
      size_t base = (size_t)rows_out[k] * D;
      touched_out[rows_out[k]] = 1;
      for (int32_t j = 0; j < D; ++j) {
        dM_out[base + j] += dO[(size_t)k * D + j];
        if (S_out != NULL) S_out[base + j] += sO[(size_t)k * D + j];
      }
    }
  }
  for (int32_t r = 0; r < V; ++r) {
    if (touched_in[r])
      for (int32_t j = 0; j < D; ++j) {
        float* m = M_in + (size_t)r * ld + j;
        *m = (float)((double)*m + dM_in[(size_t)r * D + j]);
      }
    if (touched_out[r])
      for (int32_t j = 0; j < D; ++j) {
        float* m = M_out + (size_t)r * ld + j;
        *m = (float)((double)*m + dM_out[(size_t)r * D + j]);
      }
  }
done:
  free(dM_in); free(dM_out); free(touched_in); free(touched_out);
  free(A); free(O); free(dA); free(dO); free(sA); free(sO); free(rows_in);
  free(rows_out); free(mask);
  return status;
}

int64_t oracle_train_epoch(const oracle_sampling* s, float* M_in, float* M_out,
                           int32_t V, int32_t D, int32_t ld,
                           double* loss_buckets, int32_t n_buckets) {
  if (oracle_validate_sampling(s) != 0) return -1;
  if (M_in == NULL || M_out == NULL || V <= 0 || D <= 0 || ld < D) return -1;
  if (loss_buckets != NULL && n_buckets <= 0) return -1;
  oracle_sentence sen;
  if (oracle_sentence_alloc(&sen, s->sentence_len, s->window, s->K) != 0)
    return -2;
  const int32_t w2 = 2 * s->window;
  int64_t applied = 0;
  int status = 0;
  for (int64_t sb = s->pos_begin; sb < s->pos_end && status == 0;
       sb += s->sentence_len) {
    int64_t se = sb + s->sentence_len;
    if (se > s->T) se = s->T;
    int32_t n_mb = oracle_sentence_minibatches(s, sb, se, &sen);
    for (int32_t m = 0; m < n_mb; ++m) {
      double loss = 0.0;
      int32_t n_ctx = 0;
      status = oracle_apply_minibatch(
          M_in, M_out, V, D, ld, w2, sen.ctx + (size_t)m * w2, sen.target[m],
          s->K, sen.negs + (size_t)m * s->K, sen.mask + (size_t)m * s->K,
          sen.alpha[m], &loss, &n_ctx);
      if (status != 0) break;
      if (loss_buckets != NULL) {
        int64_t b = sen.pos[m] * (int64_t)n_buckets / s->T;
        loss_buckets[2 * b] += loss;
        loss_buckets[2 * b + 1] += (double)n_ctx;
      }
      ++applied;
    }
  }
  oracle_sentence_free(&sen);
  return status == 0 ? applied : -1;
}

/*
 * Algorithm 1 (the original Hogwild SGD of word2vec, one thread), sequential.
 * For one target word and its input words in window order, each input word i
 * runs its own K+1 logistic regressions: the target (label 1) and K
 * negatives of its own (label 0; a draw equal to the target is skipped).
 * Every inner product uses the M_out row as it is at that moment (it was
 * moved by the previous pairs), the M_out row moves right after its pair,
 * and the M_in row of i moves once, after its K+1 pairs, by the sum of
 * alpha * error * (M_out row as used). Reading: the negatives of input word
 * i are the draws 2 + iK .. 2 + iK + K - 1 of the target's random stream, so
 * input word 0 draws exactly the negatives a HogBatch minibatch shares.
 * Arithmetic in fp64 from the stored fp32 values; each row update is
 * rounded to fp32 when it is written.
 */
int32_t oracle_pair_negative(const oracle_sampling* s, int64_t p, int32_t i,
                             int32_t k) {
  uint32_t word = 2u + (uint32_t)i * (uint32_t)s->K + (uint32_t)k;
  uint32_t r = oracle_draw_u32(s->seed, (uint64_t)p, (uint64_t)s->epoch, word);
  return s->neg_table[((uint64_t)r * (uint64_t)s->table_size) >> 32];
}

/* One SGD step of the logistic loss of a single (input vector, output row)
 * pair, the unit Alg. 1 works in. With x = v . u and label l (1 for the
 * target, 0 for a negative), the pair's loss is -log sigma(x) or
 * -log sigma(-x); its gradient is -(l - sigma(x)) v with respect to u and
 * -(l - sigma(x)) u with respect to v. The output row takes its step at once
 * (rounded to fp32 as it is stored); the step of the input vector is added
 * into v_step, because the input vector stays fixed until all of its word's
 * pairs have run. u is scratch. Returns the pair's loss. */
static double logistic_pair_step(const double* v, float* out_row, int32_t D,
                                 double label, double alpha, double* u,
                                 double* v_step) {
  double x = 0.0;
  for (int32_t j = 0; j < D; ++j) {
    u[j] = (double)out_row[j];
    x += v[j] * u[j];
  }
  const double coef = alpha * (label - sigma(x));
  for (int32_t j = 0; j < D; ++j) {
    v_step[j] += coef * u[j];
    out_row[j] = (float)(u[j] + coef * v[j]);
  }
  return -log_sigma(label > 0.0 ? x : -x);
}

/* The Alg. 1 update of one target word: returns -1 when an id is out of
 * range (nothing is applied), else 0, and adds the pairs' losses to *loss.
 * Input words are taken in window order. Each one pairs with the target
 * (label 1) and then with its own K draws (label 0; a draw equal to the
 * target forms no pair), every pair stepping the output row as the pairs
 * before it left it; the input word's row then moves by the sum of its
 * pairs' steps. v, u and v_step are D doubles of scratch. */
static int alg1_target(const oracle_sampling* s, float* M_in, float* M_out,
                       int32_t V, int32_t D, int32_t ld, int64_t p,
                       int32_t target, const int32_t* ctx, int32_t n,
                       float alpha, double* v, double* u, double* v_step,
                       double* loss) {
  if (target < 0 || target >= V) return -1;
  for (int32_t i = 0; i < n; ++i) {
    if (ctx[i] < 0 || ctx[i] >= V) return -1;
    for (int32_t k = 0; k < s->K; ++k) {
      int32_t neg = oracle_pair_negative(s, p, i, k);
      if (neg < 0 || neg >= V) return -1;
    }
  }
  const double a = (double)alpha;
  for (int32_t i = 0; i < n; ++i) {
    float* in_row = M_in + (size_t)ctx[i] * ld;
    for (int32_t j = 0; j < D; ++j) {
      v[j] = (double)in_row[j];
      v_step[j] = 0.0;
    }
    *loss += logistic_pair_step(v, M_out + (size_t)target * ld, D, 1.0, a, u, v_step);
    for (int32_t k = 0; k < s->K; ++k) {
      const int32_t drawn = oracle_pair_negative(s, p, i, k);
      if (drawn == target) continue;
      *loss += logistic_pair_step(v, M_out + (size_t)drawn * ld, D, 0.0, a, u, v_step);
    }
    for (int32_t j = 0; j < D; ++j) in_row[j] = (float)(v[j] + v_step[j]);
  }
  return 0;
}

int64_t oracle_pairwise_train_epoch(const oracle_sampling* s, float* M_in,
                                    float* M_out, int32_t V, int32_t D,
                                    int32_t ld, double* loss_buckets,
                                    int32_t n_buckets) {
  if (oracle_validate_sampling(s) != 0) return -1;
  if (M_in == NULL || M_out == NULL || V <= 0 || D <= 0 || ld < D) return -1;
  if (loss_buckets != NULL && n_buckets <= 0) return -1;
  oracle_sentence sen;
  if (oracle_sentence_alloc(&sen, s->sentence_len, s->window, s->K) != 0)
    return -2;
  double* v = (double*)malloc(sizeof(double) * (size_t)D);
  double* u = (double*)malloc(sizeof(double) * (size_t)D);
  double* v_step = (double*)malloc(sizeof(double) * (size_t)D);
  const int32_t w2 = 2 * s->window;
  int64_t applied = 0;
  int status = (v && u && v_step) ? 0 : -2;
  for (int64_t sb = s->pos_begin; sb < s->pos_end && status == 0;
       sb += s->sentence_len) {
    int64_t se = sb + s->sentence_len;
    if (se > s->T) se = s->T;
    int32_t n_mb = oracle_sentence_minibatches(s, sb, se, &sen);
    for (int32_t m = 0; m < n_mb; ++m) {
      double loss = 0.0;
      status = alg1_target(s, M_in, M_out, V, D, ld, sen.pos[m], sen.target[m],
                           sen.ctx + (size_t)m * w2, sen.n_ctx[m], sen.alpha[m],
                           v, u, v_step, &loss);
      if (status != 0) break;
      if (loss_buckets != NULL) {
        int64_t b = sen.pos[m] * (int64_t)n_buckets / s->T;
        loss_buckets[2 * b] += loss;
        loss_buckets[2 * b + 1] += (double)sen.n_ctx[m];
      }
      ++applied;
    }
  }
  free(v); free(u); free(v_step);
  oracle_sentence_free(&sen);
  return status == 0 ? applied : status;
}

/*
 * Negatives shared across a group of consecutive targets (a generalisation
 * of the sharing across one target's input words, Sec. 1.1). Reading: the
 * retained targets of a sentence are cut into groups of G consecutive
 * retained indices (q0 = 0, G, 2G, ...); the members of a group are those
 * that form a minibatch; all members take the K negatives drawn at the
 * group's first retained position (draws 2..K+1 of its stream; a negative
 * equal to a member's own target is masked for that member only). Every
 * member's minibatch step is computed from the rows as they were before the
 * group, and the updates of all members are summed per row in fp64 and
 * rounded once when the group ends. With G = 1 this is the HogBatch epoch.
 * The loss of a group is credited to the bucket of its first member.
 */
int64_t oracle_grouped_train_epoch(const oracle_sampling* s, int32_t G,
                                   float* M_in, float* M_out, int32_t V,
                                   int32_t D, int32_t ld, double* loss_buckets,
                                   int32_t n_buckets) {
  if (oracle_validate_sampling(s) != 0 || G < 1) return -1;
  if (M_in == NULL || M_out == NULL || V <= 0 || D <= 0 || ld < D) return -1;
  if (loss_buckets != NULL && n_buckets <= 0) return -1;
  oracle_sentence sen;
  if (oracle_sentence_alloc(&sen, s->sentence_len, s->window, s->K) != 0)
    return -2;
  const int32_t w2 = 2 * s->window;
  const int32_t K = s->K;
  const int32_t C = K + 1;
  /* all members' snapshot rows and deltas, one after another */
  double* A = (double*)malloc(sizeof(double) * (size_t)G * w2 * D);
  double* O = (double*)malloc(sizeof(double) * (size_t)G * C * D);
  double* dA = (double*)malloc(sizeof(double) * (size_t)G * w2 * D);
  double* dO = (double*)malloc(sizeof(double) * (size_t)G * C * D);
  double* acc = (double*)malloc(sizeof(double) * (size_t)D);
  int32_t* rows_in = (int32_t*)malloc(sizeof(int32_t) * (size_t)G * w2);
  int32_t* rows_out = (int32_t*)malloc(sizeof(int32_t) * (size_t)G * C);
  int32_t* negs = (int32_t*)malloc(sizeof(int32_t) * (size_t)(K + 1));
  uint8_t* mask = (uint8_t*)malloc((size_t)(K + 1));
  int32_t* q_of = (int32_t*)malloc(sizeof(int32_t) * (size_t)s->sentence_len);
  int status = (A && O && dA && dO && acc && rows_in && rows_out && negs &&
                mask && q_of) ? 0 : -2;
  int64_t applied = 0;
  for (int64_t sb = s->pos_begin; sb < s->pos_end && status == 0;
       sb += s->sentence_len) {
    int64_t se = sb + s->sentence_len;
    if (se > s->T) se = s->T;
    int32_t n_mb = oracle_sentence_minibatches(s, sb, se, &sen);
    /* retained index of every minibatch's target */
    for (int32_t m = 0, q = 0; m < n_mb; ++m) {
      while (sen.ret_pos[q] != sen.pos[m]) ++q;
      q_of[m] = q;
    }
    for (int32_t m0 = 0; m0 < n_mb && status == 0;) {
      const int32_t q0 = q_of[m0] - q_of[m0] % G;
      int32_t n_mem = 0;
      while (m0 + n_mem < n_mb && q_of[m0 + n_mem] < q0 + G) ++n_mem;
      /* the group's negatives: draws at its first retained position */
      const int64_t p0 = sen.ret_pos[q0];
      for (int32_t k = 0; k < K; ++k) {
        uint32_t r = oracle_draw_u32(s->seed, (uint64_t)p0, (uint64_t)s->epoch,
                                     2u + (uint32_t)k);
        negs[k] = s->neg_table[((uint64_t)r * (uint64_t)s->table_size) >> 32];
        if (negs[k] < 0 || negs[k] >= V) status = -1;
      }
      if (status != 0) break;
      double loss = 0.0;
      int32_t n_in = 0;  /* input rows of all members so far */
      for (int32_t g = 0; g < n_mem; ++g) {
        const int32_t m = m0 + g;
        const int32_t n = sen.n_ctx[m];
        const int32_t* ctx = sen.ctx + (size_t)m * w2;
        for (int32_t i = 0; i < n; ++i) {
          if (ctx[i] < 0 || ctx[i] >= V) status = -1;
          rows_in[n_in + i] = ctx[i];
        }
        if (status != 0) break;
        for (int32_t i = 0; i < n; ++i)
          for (int32_t j = 0; j < D; ++j)
            A[((size_t)n_in + i) * D + j] = (double)M_in[(size_t)ctx[i] * ld + j];
        for (int32_t k = 0; k <= K; ++k) {
          const int32_t id = k == 0 ? sen.target[m] : negs[k - 1];
          rows_out[g * C + k] = id;
          for (int32_t j = 0; j < D; ++j)
            O[((size_t)g * C + k) * D + j] = (double)M_out[(size_t)id * ld + j];
        }
        for (int32_t k = 0; k < K; ++k) mask[k] = (uint8_t)(negs[k] == sen.target[m]);
        double l = 0.0;
        oracle_sgns_delta(n, K, D, A + (size_t)n_in * D, O + (size_t)g * C * D,
                          mask, (double)sen.alpha[m], NULL, dA + (size_t)n_in * D,
                          dO + (size_t)g * C * D, &l);
        loss += l;
        n_in += n;
      }
      if (status != 0) break;
      /* every member read the rows as they were before the group; the sums
       * per row are rounded once */
      write_back(M_in, D, ld, n_in, rows_in, dA, acc);
      write_back(M_out, D, ld, n_mem * C, rows_out, dO, acc);
      if (loss_buckets != NULL) {
        int64_t b = sen.pos[m0] * (int64_t)n_buckets / s->T;
        loss_buckets[2 * b] += loss;
        loss_buckets[2 * b + 1] += (double)n_in;
      }
      applied += n_mem;
      m0 += n_mem;
    }
  }
  free(A); free(O); free(dA); free(dO); free(acc); free(rows_in); free(rows_out);
  free(negs); free(mask); free(q_of);
  oracle_sentence_free(&sen);
  return status == 0 ? applied : status;
}
