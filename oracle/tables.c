/*
 * Oracle: sampling tables. TEST INFRASTRUCTURE ONLY.
 *
 * The paper trains with "negative samples=5" and "sample=1e-4" (Sec. 2,
 * hyper-parameters) and draws each negative as "one word from V" (Alg. 1), but
 * prints neither the negative distribution nor the subsampling rule. Readings
 * taken here (both stated as formulas, both exact integer decisions):
 *   - negatives follow the unigram distribution raised to `neg_power` (0.75),
 *     discretised into a table of `table_size` slots by floor of the
 *     normalised prefix sums;
 *   - a word of relative frequency f is kept with probability
 *     min(1, sqrt(t/f) + t/f), encoded as a uint32 threshold.
 */
#include <math.h>
#include <stdlib.h>

#include "oracle.h"

int oracle_build_tables(const int64_t* counts, int32_t V, double neg_power,
                        double sample_t, int32_t* neg_table, int64_t table_size,
                        uint32_t* keep_thresh) {
  if (counts == NULL || V <= 0) return -1;
  if (neg_table != NULL && (table_size <= 0 || table_size >= (1LL << 32)))
    return -1;
  if (sample_t < 0.0) return -1;
  int64_t total = 0;
  for (int32_t w = 0; w < V; ++w) {
    if (counts[w] < 0) return -1;
    total += counts[w];
  }
  if (total <= 0) return -1;

  if (neg_table != NULL) {
    /* Unnormalised weights and their running sums, left to right in fp64. */
    double* prefix = (double*)malloc(sizeof(double) * (size_t)V);
    if (prefix == NULL) return -2;
    double run = 0.0;
    for (int32_t w = 0; w < V; ++w) {
      run += pow((double)counts[w], neg_power);
      prefix[w] = run;
    }
    double last = prefix[V - 1];
    int64_t begin = 0;
    for (int32_t w = 0; w < V; ++w) {
      int64_t end = (w == V - 1)
                        ? table_size
                        : (int64_t)floor(prefix[w] / last * (double)table_size);
      if (end > table_size) end = table_size;
      for (int64_t s = begin; s < end; ++s) neg_table[s] = w;
      if (end > begin) begin = end;
    }
    free(prefix);
  }

  if (keep_thresh != NULL) {
    for (int32_t w = 0; w < V; ++w) {
      if (sample_t == 0.0 || counts[w] == 0) {
        keep_thresh[w] = 0xFFFFFFFFu;
        continue;
      }
      double f = (double)counts[w] / (double)total;
      double ratio = sample_t / f;
      double p_keep = sqrt(ratio) + ratio;
      if (p_keep >= 1.0) {
        keep_thresh[w] = 0xFFFFFFFFu;
      } else {
        double scaled = floor(p_keep * 4294967296.0);
        keep_thresh[w] = scaled >= 1.0 ? (uint32_t)(scaled - 1.0) : 0u;
      }
    }
  }
  return 0;
}
