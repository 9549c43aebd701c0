// Host construction of the sampling tables (negative table, keep thresholds).
//
// The paper trains with 5 negatives and sample = 1e-4 (Sec. 2) and draws each
// negative "from V" (Alg. 1) without printing the distributions; the readings
// implemented here are stated in include/w2v.h: unigram^power negatives
// discretised by floor of normalised fp64 prefix sums, and keep probability
// min(1, sqrt(t/f) + t/f) encoded as a uint32 threshold. Pure integer
// decisions downstream make GPU sampling reproducible bit for bit.
#include <math.h>
#include <stdint.h>

#include <vector>

#include "w2v_internal.h"

namespace w2v {

int build_tables(const int64_t* counts, int32_t V, double power,
                 double sample_t, int32_t* table, int64_t table_size,
                 uint32_t* keep) {
  if (counts == nullptr) return fail(W2V_EINVAL, "counts is NULL");
  if (V <= 0) return fail(W2V_EINVAL, "V must be positive");
  if (table != nullptr && (table_size <= 0 || table_size >= (int64_t(1) << 32)))
    return fail(W2V_EINVAL, "table_size must be in [1, 2^32)");
  if (!(sample_t >= 0.0)) return fail(W2V_EINVAL, "sample_t must be >= 0");
  int64_t total = 0;
  for (int32_t w = 0; w < V; ++w) {
    if (counts[w] < 0) return fail(W2V_EINVAL, "negative count");
    total += counts[w];
  }
  if (total <= 0) return fail(W2V_EINVAL, "counts sum to zero");

  if (table != nullptr) {
    std::vector<double> run;
    try {
      run.resize((size_t)V);
    } catch (...) {
      return fail(W2V_ENOMEM, "host allocation failed");
    }
    double acc = 0.0;
    for (int32_t w = 0; w < V; ++w) {
      acc += pow((double)counts[w], power);
      run[(size_t)w] = acc;
    }
    const double norm = run[(size_t)V - 1];
    int64_t slot = 0;
    for (int32_t w = 0; w < V; ++w) {
      int64_t bound = table_size;
      if (w != V - 1) {
        bound = (int64_t)floor(run[(size_t)w] / norm * (double)table_size);
        if (bound > table_size) bound = table_size;
      }
      while (slot < bound) table[slot++] = w;
    }
  }

  if (keep != nullptr) {
    for (int32_t w = 0; w < V; ++w) {
      if (sample_t == 0.0 || counts[w] == 0) {
        keep[w] = 0xFFFFFFFFu;
        continue;
      }
      const double f = (double)counts[w] / (double)total;
      const double r = sample_t / f;
      const double p = sqrt(r) + r;
      if (p >= 1.0) {
        keep[w] = 0xFFFFFFFFu;
      } else {
        const double top = floor(p * 4294967296.0);
        keep[w] = top >= 1.0 ? (uint32_t)(top - 1.0) : 0u;
      }
    }
  }
  return ok();
}

int hot_rows(const int64_t* counts, int32_t V, double power, double sample_t,
             int32_t window, int32_t K, int64_t inflight, double tol) {
  if (counts == nullptr) return fail(W2V_EINVAL, "counts is NULL");
  if (V <= 0) return fail(W2V_EINVAL, "V must be positive");
  if (window < 1 || K < 0) return fail(W2V_EINVAL, "need window >= 1, K >= 0");
  if (inflight < 1) return fail(W2V_EINVAL, "inflight must be >= 1");
  if (!(tol > 0.0)) return fail(W2V_EINVAL, "tol must be positive");
  if (!(sample_t >= 0.0)) return fail(W2V_EINVAL, "sample_t must be >= 0");
  int64_t total = 0;
  for (int32_t w = 0; w < V; ++w) {
    if (counts[w] < 0) return fail(W2V_EINVAL, "negative count");
    total += counts[w];
  }
  if (total <= 0) return fail(W2V_EINVAL, "counts sum to zero");
  // Kept mass per word and negative-sampling weight per word.
  double kept_sum = 0.0, neg_sum = 0.0;
  std::vector<double> kept((size_t)V), negw((size_t)V);
  for (int32_t w = 0; w < V; ++w) {
    const double c = (double)counts[w];
    double p = 1.0;
    if (sample_t > 0.0 && counts[w] > 0) {
      const double r = sample_t / (c / (double)total);
      p = sqrt(r) + r;
      if (p > 1.0) p = 1.0;
    }
    kept[(size_t)w] = c * p;
    negw[(size_t)w] = pow(c, power);
    kept_sum += kept[(size_t)w];
    neg_sum += negw[(size_t)w];
  }
  const double others = (double)(inflight - 1);
  int32_t H = 0;
  for (int32_t w = 0; w < V; ++w) {
    const double rho = kept[(size_t)w] / kept_sum;
    const double q = negw[(size_t)w] / neg_sum;
    const double p_out = rho + (double)K * q;
    const double p_in = (double)(window + 1) * rho;
    const double p = p_out > p_in ? p_out : p_in;
    if (others * p >= tol) H = w + 1;
  }
  ok();
  return H;
}

}  // namespace w2v
