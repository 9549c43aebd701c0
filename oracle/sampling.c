/*
 * Oracle: formation of HogBatch minibatches from a corpus. TEST
 * INFRASTRUCTURE ONLY.
 *
 * One minibatch is "1 target word w_out^t and N input words" (Alg. 1 header)
 * together with K negatives shared by all N input words (Sec. 1.1, negative
 * sample sharing). The paper fixes window = 5, negative = 5, sample = 1e-4
 * (Sec. 2) but not the sentence, window or learning-rate rules. Readings:
 *   - the corpus is cut into sentences of sentence_len raw tokens; windows
 *     never cross a sentence;
 *   - subsampling is decided per raw position before windows are formed;
 *   - the retained word at retained index q is a target; its half-width is
 *     h = w - b with b uniform on {0..w-1}; its input words are the retained
 *     words at retained indices q-h..q+h other than q, in increasing order;
 *   - a target with no input word forms no minibatch;
 *   - negatives are K table draws; a draw equal to the target is masked;
 *   - the learning rate decays linearly in the raw position over all epochs
 *     to a floor of min_alpha_frac * alpha0, computed in fp64, rounded once;
 *   - every random decision is the draw of oracle_draw_u32 at the target's
 *     raw position: word 0 keep, word 1 window, words 2..K+1 negatives, each
 *     mapped to a range by the multiply-shift floor(r * n / 2^32).
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include "oracle.h"
#include "oracle_internal.h"

int oracle_validate_sampling(const oracle_sampling* s) {
  if (s == NULL || s->corpus == NULL || s->neg_table == NULL) return -1;
  if (s->T <= 0 || s->sentence_len <= 0) return -1;
  if (s->window <= 0 || s->K < 0) return -1;
  if (s->table_size <= 0 || s->table_size >= (1LL << 32)) return -1;
  if (s->n_epochs <= 0 || s->epoch < 0 || s->epoch >= s->n_epochs) return -1;
  if (s->pos_begin < 0 || s->pos_end > s->T || s->pos_begin > s->pos_end)
    return -1;
  if (s->pos_begin % s->sentence_len != 0) return -1;
  if (s->pos_end != s->T && s->pos_end % s->sentence_len != 0) return -1;
  return 0;
}

float oracle_alpha_at(const oracle_sampling* s, int64_t p) {
  double done = (double)s->epoch * (double)s->T + (double)p;
  double all = (double)s->n_epochs * (double)s->T;
  double frac = 1.0 - done / all;
  double floor_frac = (double)s->min_alpha_frac;
  if (frac < floor_frac) frac = floor_frac;
  double a = (double)s->alpha0 * frac;
  return (float)a;
}

/* floor(r * n / 2^32) for a 32-bit draw r and a range n < 2^32. */
static uint64_t scale_draw(uint32_t r, uint64_t n) {
  return ((uint64_t)r * n) >> 32;
}

int32_t oracle_sentence_minibatches(const oracle_sampling* s, int64_t sb,
                                    int64_t se, oracle_sentence* out) {
  const uint64_t e = (uint64_t)s->epoch;
  const int32_t w = s->window;
  /* Subsampling decision per raw position, then compaction. */
  int32_t n_ret = 0;
  for (int64_t p = sb; p < se; ++p) {
    int keep = 1;
    if (s->keep_thresh != NULL) {
      uint32_t r = oracle_draw_u32(s->seed, (uint64_t)p, e, 0);
      keep = r <= s->keep_thresh[s->corpus[p]];
    }
    if (keep) out->ret_pos[n_ret++] = p;
  }
  int32_t n_mb = 0;
  for (int32_t q = 0; q < n_ret; ++q) {
    int64_t p = out->ret_pos[q];
    int32_t target = s->corpus[p];
    uint32_t rb = oracle_draw_u32(s->seed, (uint64_t)p, e, 1);
    int32_t h = w - (int32_t)scale_draw(rb, (uint64_t)w);
    int32_t* ctx = out->ctx + (size_t)n_mb * 2 * w;
    int32_t n = 0;
    for (int32_t j = q - h; j <= q + h; ++j) {
      if (j == q || j < 0 || j >= n_ret) continue;
      ctx[n++] = s->corpus[out->ret_pos[j]];
    }
    if (n == 0) continue;
    for (int32_t i = n; i < 2 * w; ++i) ctx[i] = -1;
    int32_t* negs = out->negs + (size_t)n_mb * s->K;
    uint8_t* mask = out->mask + (size_t)n_mb * s->K;
    for (int32_t k = 0; k < s->K; ++k) {
      uint32_t r = oracle_draw_u32(s->seed, (uint64_t)p, e, 2u + (uint32_t)k);
      int32_t neg = s->neg_table[scale_draw(r, (uint64_t)s->table_size)];
      negs[k] = neg;
      mask[k] = (uint8_t)(neg == target);
    }
    out->target[n_mb] = target;
    out->n_ctx[n_mb] = n;
    out->alpha[n_mb] = oracle_alpha_at(s, p);
    out->pos[n_mb] = p;
    ++n_mb;
  }
  return n_mb;
}

int oracle_sentence_alloc(oracle_sentence* o, int32_t sentence_len,
                          int32_t window, int32_t K) {
  size_t L = (size_t)sentence_len;
  o->ret_pos = (int64_t*)malloc(sizeof(int64_t) * L);
  o->pos = (int64_t*)malloc(sizeof(int64_t) * L);
  o->target = (int32_t*)malloc(sizeof(int32_t) * L);
  o->n_ctx = (int32_t*)malloc(sizeof(int32_t) * L);
  o->ctx = (int32_t*)malloc(sizeof(int32_t) * L * 2 * (size_t)window);
  o->negs = (int32_t*)malloc(sizeof(int32_t) * (L * (size_t)K + 1));
  o->mask = (uint8_t*)malloc(L * (size_t)K + 1);
  o->alpha = (float*)malloc(sizeof(float) * L);
  if (!o->ret_pos || !o->pos || !o->target || !o->n_ctx || !o->ctx ||
      !o->negs || !o->mask || !o->alpha) {
    oracle_sentence_free(o);
    return -2;
  }
  return 0;
}

void oracle_sentence_free(oracle_sentence* o) {
  free(o->ret_pos); free(o->pos); free(o->target); free(o->n_ctx);
  free(o->ctx); free(o->negs); free(o->mask); free(o->alpha);
  memset(o, 0, sizeof(*o));
}

int64_t oracle_minibatches(const oracle_sampling* s, int32_t* out_targets,
                           int32_t* out_ctx, int32_t* out_negs,
                           uint8_t* out_mask, float* out_alpha,
                           int64_t* out_pos, int64_t cap) {
  if (oracle_validate_sampling(s) != 0 || cap < 0) return -1;
  oracle_sentence sen;
  if (oracle_sentence_alloc(&sen, s->sentence_len, s->window, s->K) != 0)
    return -2;
  const int32_t w2 = 2 * s->window;
  int64_t total = 0;
  for (int64_t sb = s->pos_begin; sb < s->pos_end; sb += s->sentence_len) {
    int64_t se = sb + s->sentence_len;
    if (se > s->T) se = s->T;
    int32_t n_mb = oracle_sentence_minibatches(s, sb, se, &sen);
    for (int32_t m = 0; m < n_mb; ++m, ++total) {
      if (total >= cap) continue;
      if (out_targets) out_targets[total] = sen.target[m];
      if (out_ctx)
        memcpy(out_ctx + total * w2, sen.ctx + (size_t)m * w2,
               sizeof(int32_t) * (size_t)w2);
      if (out_negs && s->K > 0)
        memcpy(out_negs + total * s->K, sen.negs + (size_t)m * s->K,
               sizeof(int32_t) * (size_t)s->K);
      if (out_mask && s->K > 0)
        memcpy(out_mask + total * s->K, sen.mask + (size_t)m * s->K,
               (size_t)s->K);
      if (out_alpha) out_alpha[total] = sen.alpha[m];
      if (out_pos) out_pos[total] = sen.pos[m];
    }
  }
  oracle_sentence_free(&sen);
  return total;
}
