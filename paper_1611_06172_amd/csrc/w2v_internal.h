// Host-side internals of libw2v: error state and shared helpers.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "w2v.h"

namespace w2v {

// Records `msg` as this thread's last error and returns `code`.
int fail(int code, const char* msg);
// Formats a message (printf-style) and records it.
int failf(int code, const char* fmt, ...);
// Clears this thread's last error and returns W2V_OK.
int ok();

int hot_rows(const int64_t* counts, int32_t V, double power, double sample_t,
             int32_t window, int32_t K, int64_t inflight, double tol);

int build_tables(const int64_t* counts, int32_t V, double power,
                 double sample_t, int32_t* table, int64_t table_size,
                 uint32_t* keep);

// Workspace of w2v_build_vocab: the vocabulary arrays and the sort's
// temporaries, plus the binned corpus, its segment table and the per-unit
// partial counts where the ids are counted by bins (vocab.hip).
size_t vocab_workspace_bytes(int32_t V, int64_t T);

}  // namespace w2v
