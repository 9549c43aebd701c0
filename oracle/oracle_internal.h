/* Oracle internals shared between the oracle's own source files only.
 * TEST INFRASTRUCTURE ONLY. */
#ifndef W2V_ORACLE_INTERNAL_H
#define W2V_ORACLE_INTERNAL_H

#include "oracle.h"

/* The minibatches of one sentence, in processing order. */
typedef struct {
  int64_t* ret_pos; /* raw positions of the retained words */
  int64_t* pos;     /* [m] raw position of the target */
  int32_t* target;  /* [m] */
  int32_t* n_ctx;   /* [m] number of input words */
  int32_t* ctx;     /* [m][2w], -1 padded */
  int32_t* negs;    /* [m][K] */
  uint8_t* mask;    /* [m][K] */
  float* alpha;     /* [m] */
} oracle_sentence;

int oracle_validate_sampling(const oracle_sampling* s);
float oracle_alpha_at(const oracle_sampling* s, int64_t p);
int oracle_sentence_alloc(oracle_sentence* o, int32_t sentence_len,
                          int32_t window, int32_t K);
void oracle_sentence_free(oracle_sentence* o);
int32_t oracle_sentence_minibatches(const oracle_sampling* s, int64_t sb,
                                    int64_t se, oracle_sentence* out);

#endif
