/*
 * Drives every entry point of the CPU oracle on small inputs (ragged
 * sentences, subsampling, the largest window and K, absent inputs, masked
 * and repeated negatives, sub-ranges, loss buckets) so that a build with
 * AddressSanitizer and UndefinedBehaviorSanitizer reports any out-of-bounds
 * access, leak, overflow or other undefined behaviour. Test infrastructure:
 * built and run by tests/test_sanitize.py. Exit status 0 when every call
 * returned what the oracle's contract says.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "oracle.h"

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;

static uint64_t next_u64(void) {
  uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

/* id with probability roughly proportional to 1 / (id + 1) */
static int32_t zipfish(int32_t V) {
  const double u = (double)(next_u64() >> 11) / 9007199254740992.0;
  int32_t id = (int32_t)floor(pow((double)V + 1.0, u)) - 1;
  return id < 0 ? 0 : (id >= V ? V - 1 : id);
}

#define CHECK(cond)                                              \
  do {                                                           \
    if (!(cond)) {                                               \
      fprintf(stderr, "check failed: %s (line %d)\n", #cond, __LINE__); \
      return 1;                                                  \
    }                                                            \
  } while (0)

int main(void) {
  const int32_t V = 97, D = 13, ld = 16;
  const int64_t T = 2 * 1024 + 777, table_size = 10007;
  int32_t* corpus = malloc(sizeof(int32_t) * T);
  int64_t* counts = calloc(V, sizeof(int64_t));
  for (int64_t i = 0; i < T; ++i) {
    corpus[i] = zipfish(V);
    counts[corpus[i]]++;
  }
  int32_t* table = malloc(sizeof(int32_t) * table_size);
  uint32_t* thr = malloc(sizeof(uint32_t) * V);
  CHECK(oracle_build_tables(counts, V, 0.75, 1e-2, table, table_size, thr) == 0);
  CHECK(oracle_build_tables(counts, V, 0.75, 0.0, NULL, 0, thr) == 0);
  CHECK(oracle_build_tables(counts, -1, 0.75, 0.0, table, table_size, thr) < 0);

  uint64_t ctr[4] = {1, 2, 3, ~0ull}, key[2] = {5, 6}, out[4];
  oracle_philox4x64_10(ctr, key, out);
  (void)oracle_draw_u32(7, 123456789, 3, 17);

  float* M_in = malloc(sizeof(float) * V * ld);
  float* M_out = malloc(sizeof(float) * V * ld);
  const int windows[3] = {1, 5, 16}, Ks[3] = {0, 5, 64}, lens[3] = {7, 1000, 1024};
  for (int c = 0; c < 3; ++c) {
    oracle_sampling s;
    memset(&s, 0, sizeof(s));
    s.corpus = corpus;
    s.T = T;
    s.pos_begin = 0;
    s.pos_end = T;
    s.sentence_len = lens[c];
    s.window = windows[c];
    s.K = Ks[c];
    s.neg_table = table;
    s.table_size = table_size;
    s.keep_thresh = c == 1 ? NULL : thr;
    s.alpha0 = 0.025f;
    s.min_alpha_frac = 1e-4f;
    s.epoch = c;
    s.n_epochs = 3;
    s.seed = 11 + c;
    const int64_t n = oracle_minibatches(&s, NULL, NULL, NULL, NULL, NULL, NULL, 0);
    CHECK(n > 0);
    const int w2 = 2 * s.window, K = s.K > 0 ? s.K : 1;
    int32_t* tg = malloc(sizeof(int32_t) * n);
    int32_t* ctx = malloc(sizeof(int32_t) * n * w2);
    int32_t* negs = malloc(sizeof(int32_t) * n * K);
    uint8_t* mask = malloc(n * K);
    float* alpha = malloc(sizeof(float) * n);
    int64_t* pos = malloc(sizeof(int64_t) * n);
    CHECK(oracle_minibatches(&s, tg, ctx, negs, mask, alpha, pos, n) == n);
    CHECK(oracle_minibatches(&s, tg, ctx, negs, mask, alpha, pos, n / 2) == n);

    for (int64_t i = 0; i < (int64_t)V * ld; ++i) {
      M_in[i] = (float)((double)(next_u64() >> 11) / 9007199254740992.0 - 0.5) / D;
      M_out[i] = 0.f;
    }
    double buckets[2 * 5];
    memset(buckets, 0, sizeof(buckets));
    CHECK(oracle_train_epoch(&s, M_in, M_out, V, D, ld, buckets, 5) == n);
    CHECK(oracle_pairwise_train_epoch(&s, M_in, M_out, V, D, ld, buckets, 5) > 0);
    for (int G = 1; G <= 8; G *= 2)
      CHECK(oracle_grouped_train_epoch(&s, G, M_in, M_out, V, D, ld, NULL, 0) > 0);
    (void)oracle_pair_negative(&s, pos[0], 1, 0);
    s.pos_begin = lens[c];
    s.pos_end = T;
    CHECK(oracle_train_epoch(&s, M_in, M_out, V, D, ld, NULL, 0) >= 0);
    for (int64_t i = 0; i < (int64_t)V * ld; ++i) CHECK(isfinite(M_in[i]) && isfinite(M_out[i]));
    free(tg), free(ctx), free(negs), free(mask), free(alpha), free(pos);
  }

  /* one minibatch and its scaled variant, with an absent input, a repeated
   * input and a masked column */
  {
    const int32_t N = 4, K = 3;
    double A[4 * 13], O[4 * 13], X[16], dA[4 * 13], dO[4 * 13], sA[4 * 13], sO[4 * 13], loss;
    for (int i = 0; i < 4 * 13; ++i) {
      A[i] = (double)(i % 7) / 10.0 - 0.3;
      O[i] = (double)(i % 5) / 10.0 - 0.2;
    }
    const uint8_t m[3] = {0, 1, 0};
    oracle_sgns_delta(N, K, D, A, O, m, 0.05, X, dA, dO, &loss);
    oracle_sgns_delta_scaled(N, K, D, A, O, m, 0.05, NULL, dA, dO, NULL, sA, sO);
    const int32_t c4[4] = {3, -1, 3, 9}, n3[3] = {2, 5, 2};
    int32_t n_ctx = 0;
    CHECK(oracle_apply_minibatch(M_in, M_out, V, D, ld, N, c4, 5, K, n3, m, 0.02f,
                                 &loss, &n_ctx) == 0);
    CHECK(n_ctx == 3);
  }

  /* snapshot batch with per-minibatch alpha and scales */
  {
    const int32_t B = 300, N = 10, K = 5;
    int32_t* t = malloc(sizeof(int32_t) * B);
    int32_t* c = malloc(sizeof(int32_t) * B * N);
    int32_t* ng = malloc(sizeof(int32_t) * B * K);
    float* al = malloc(sizeof(float) * B);
    for (int b = 0; b < B; ++b) {
      t[b] = zipfish(V);
      al[b] = 0.001f * (float)(1 + b % 7);
      for (int i = 0; i < N; ++i) c[b * N + i] = (next_u64() % 5 == 0) ? -1 : zipfish(V);
      for (int k = 0; k < K; ++k) ng[b * K + k] = zipfish(V);
    }
    double* S_in = malloc(sizeof(double) * V * D);
    double* S_out = malloc(sizeof(double) * V * D);
    CHECK(oracle_step_batch(B, N, K, t, c, ng, al, 0.f, M_in, M_out, V, D, ld, S_in,
                            S_out) == 0);
    CHECK(oracle_step_batch(B, N, K, t, c, ng, NULL, 0.01f, M_in, M_out, V, D, ld, NULL,
                            NULL) == 0);
    free(t), free(c), free(ng), free(al), free(S_in), free(S_out);
  }
  free(corpus), free(counts), free(table), free(thr), free(M_in), free(M_out);
  puts("oracle sanitizer check: ok");
  return 0;
}
