// Drives the GPU library's host-side table construction and conflict model
// (csrc/tables.cpp: w2v::build_tables, w2v::hot_rows) on edge-case inputs so
// that a build with AddressSanitizer and UndefinedBehaviorSanitizer reports
// any out-of-bounds access, leak or undefined behaviour. The error-recording
// helpers of csrc/api.hip are replaced by the minimal ones below (the HIP
// side is not built here). Test infrastructure: built and run by
// tests/test_sanitize.py; exit status 0 when every call returned what the
// header documents.
#include <math.h>
#include <stdint.h>
#include <stdio.h>

#include <vector>

#include "w2v_internal.h"

namespace w2v {
int fail(int code, const char*) { return code; }
int failf(int code, const char*, ...) { return code; }
int ok() { return W2V_OK; }
}  // namespace w2v

#define CHECK(cond)                                                      \
  do {                                                                   \
    if (!(cond)) {                                                       \
      fprintf(stderr, "check failed: %s (line %d)\n", #cond, __LINE__); \
      return 1;                                                          \
    }                                                                    \
  } while (0)

int main() {
  for (int32_t V : {1, 2, 1000, 100003}) {
    std::vector<int64_t> c(V);
    for (int32_t w = 0; w < V; ++w) c[w] = (int64_t)(1e7 / (w + 1.0)) + (w % 3 == 0 ? 0 : 1);
    if (V > 2) c[V / 2] = 0;  // a word that never occurs
    for (int64_t ts : {(int64_t)1, (int64_t)V, (int64_t)10007, (int64_t)1000000}) {
      std::vector<int32_t> table(ts);
      std::vector<uint32_t> keep(V);
      CHECK(w2v::build_tables(c.data(), V, 0.75, 1e-4, table.data(), ts, keep.data()) ==
            W2V_OK);
      for (int64_t i = 0; i < ts; ++i) CHECK(table[i] >= 0 && table[i] < V);
      CHECK(w2v::build_tables(c.data(), V, 1.0, 0.0, nullptr, 0, keep.data()) == W2V_OK);
      CHECK(w2v::build_tables(c.data(), V, 0.0, 1.0, table.data(), ts, nullptr) == W2V_OK);
    }
    for (int64_t inflight : {(int64_t)1, (int64_t)64, (int64_t)2048, (int64_t)1 << 40})
      for (double tol : {0.05, 0.5, 128.0}) {
        const int h = w2v::hot_rows(c.data(), V, 0.75, 1e-4, 5, 5, inflight, tol);
        CHECK(h >= 0 && h <= V);
      }
  }
  std::vector<int64_t> zero(10, 0), neg(10, 1);
  neg[3] = -1;
  std::vector<int32_t> t(8);
  CHECK(w2v::build_tables(zero.data(), 10, 0.75, 0.0, t.data(), 8, nullptr) == W2V_EINVAL);
  CHECK(w2v::build_tables(neg.data(), 10, 0.75, 0.0, t.data(), 8, nullptr) == W2V_EINVAL);
  CHECK(w2v::build_tables(nullptr, 10, 0.75, 0.0, t.data(), 8, nullptr) == W2V_EINVAL);
  CHECK(w2v::build_tables(neg.data(), 10, 0.75, NAN, t.data(), 8, nullptr) == W2V_EINVAL);
  CHECK(w2v::hot_rows(nullptr, 10, 0.75, 1e-4, 5, 5, 64, 0.5) < 0);
  puts("host tables sanitizer check: ok");
  return 0;
}
