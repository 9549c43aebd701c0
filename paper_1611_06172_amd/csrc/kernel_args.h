// Argument blocks of the HogBatch kernels and their host launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace w2v {

// Sentence-parallel epoch (training or minibatch export).
struct EpochArgs {
  const int32_t* corpus;
  int64_t T, pos_begin, pos_end;
  int64_t n_sent;          // sentences in [pos_begin, pos_end)
  int32_t L;               // sentence length
  float* M_in;
  float* M_out;
  int32_t V, D;
  int64_t ld;
  int32_t w, K;
  const int32_t* table;
  int64_t table_size;
  const uint32_t* thr;     // NULL: keep every position
  float alpha0, min_frac;
  int32_t epoch, n_epochs;
  uint64_t seed;
  double* loss;            // NULL or double[2 * n_buckets]
  int32_t n_buckets;
  int64_t* stats;          // NULL or int64[5]
  int32_t* status;         // NULL or the device's error word (host-mapped)
  int32_t hot_rows;        // ids below this get atomic updates
  int32_t split_rows;      // ids below this use partial rows in `part`
  int32_t group;           // consecutive targets sharing one negative draw
  float* part;             // [2][split_rows][kSplitParts][ld] partial rows
  int32_t pend_slots;      // LDS pending input-row slots per wavefront (0: none)
  int32_t pend_from;       // ids below this never take a pending slot
  int32_t target_batch;    // targets k_epoch forms at once (<= 64; its
                           // negatives take target_batch * K ints of LDS)
  // export outputs (minibatch export only)
  int32_t* out_targets;
  int32_t* out_ctx;
  int32_t* out_negs;
  uint8_t* out_mask;
  float* out_alpha;
};

// Snapshot batch of independent minibatches.
struct StepArgs {
  int32_t B, N, K;
  const int32_t* targets;
  const int32_t* contexts;
  const int32_t* negatives;
  const float* alpha;      // NULL: alpha_scalar
  float alpha_scalar;
  float* M_in;             // rows read, then updated by the finalize pass
  float* M_out;
  double* dM_in;           // fp64 delta buffers (workspace), row stride ld
  double* dM_out;
  int32_t V, D;
  int64_t ld;
  int64_t* stats;
  int32_t* status;         // NULL or the device's error word (host-mapped)
};

// Sorted snapshot batch: the snapshot batch's inputs plus the staging rows
// and sort keys it writes (step_sorted.hip sets the workspace pointers).
struct SortedStepArgs {
  int32_t B, N, K;
  const int32_t* targets;
  const int32_t* contexts;
  const int32_t* negatives;
  const float* alpha;      // NULL: alpha_scalar
  float alpha_scalar;
  float* M_in;
  float* M_out;
  int32_t V, D;
  int64_t ld;
  int64_t* stats;
  int32_t* status;         // NULL or the device's error word (host-mapped)
  float* stage_in;         // [B][N][ld] updates of the distinct input rows
  float* stage_out;        // [B][K+1][ld] updates of the output rows
  uint32_t* key_in;        // [B][N] sort key of each staging row: the M_in
                           // row id, 2V if unused
  int32_t* val_in;         // [B][N] staging index
  uint32_t* key_out;       // [B][K+1] V + the M_out row id, 2V if unused
  int32_t* val_out;        // [B][K+1] staging index (counted from stage_in)
  int64_t out_base;        // staging index of stage_out's first row
};

// Workgroups of one wavefront of `kernel` resident per CU with `dyn_lds`
// bytes of dynamic LDS (0 on a failed query).
int resident_blocks_per_cu(const void* kernel, size_t dyn_lds);

// Launchers (defined next to the kernels). Return a hipError_t.
// C: columns per lane (D <= 64 C); nmax: max input words per minibatch.
hipError_t launch_train(int C, int nmax, const EpochArgs& a, int grid,
                        hipStream_t s);
hipError_t launch_export(const EpochArgs& a, int grid, hipStream_t s);
// Clears the partial rows / adds them into M_in, M_out and clears them.
hipError_t launch_part_clear(const EpochArgs& a, hipStream_t s);
hipError_t launch_part_fold(const EpochArgs& a, hipStream_t s);
hipError_t launch_step(int C, int nmax, const StepArgs& a, int grid,
                       hipStream_t s);
bool train_shape_supported(int C, int nmax);
// Sorted snapshot batch (step_sorted.hip).
size_t sorted_step_workspace_bytes(int32_t B, int32_t N, int32_t K, int32_t V,
                                   int32_t ld);
bool sorted_step_supported(int C, int nmax);
hipError_t launch_step_sorted(int C, int nmax, SortedStepArgs a, void* workspace,
                              hipStream_t s);
int columns_for(int D);      // compiled C for a row length, 0 if none
int inputs_cap_for(int n);   // compiled nmax for n input words, 0 if none
int train_blocks_per_cu(int C, int nmax, int K);
// Pending input-row slots that fit beside the training kernel's LDS without
// lowering its occupancy (0 if fewer than two fit).
int train_pending_slots(int C, int nmax, int K);
// Targets the training kernel forms at once: 64, or fewer where the
// negatives of 64 targets would cost LDS residency (large K).
int train_target_batch(int C, int nmax, int K);
// HogBatch with negatives shared by groups of targets: omax = compiled
// capacity of output columns (G + K).
int group_outputs_cap_for(int n);
bool grouped_shape_supported(int C, int omax);
int grouped_blocks_per_cu(int C, int omax, int K);
hipError_t launch_grouped(int C, int omax, const EpochArgs& a, int grid,
                          hipStream_t s);
// Vocabulary of a raw id stream (vocab.hip).
size_t vocab_workspace_bytes(int32_t V);
hipError_t launch_vocab(const int32_t* raw, int64_t T, int32_t V,
                        int64_t min_count, int64_t* ranked_counts,
                        int32_t* rank_of, int32_t* v_kept, int32_t* corpus_out,
                        void* workspace, hipStream_t s);
// Stable LSD radix sort of (key, value) pairs, keys < 2^bits (radix_sort.hip);
// vals_in NULL means values 0..n-1. temp: radix_sort_temp_bytes(n,
// sizeof(key)) bytes, 256-byte aligned; keys_out/vals_out must not overlap
// the inputs or temp.
size_t radix_sort_temp_bytes(int64_t n, size_t key_bytes);
hipError_t radix_sort_pairs(const uint32_t* keys_in, const int32_t* vals_in,
                            uint32_t* keys_out, int32_t* vals_out, int64_t n,
                            int bits, void* temp, hipStream_t s);
hipError_t radix_sort_pairs(const unsigned long long* keys_in, const int32_t* vals_in,
                            unsigned long long* keys_out, int32_t* vals_out, int64_t n,
                            int bits, void* temp, hipStream_t s);
// Algorithm 1 (per-pair) epoch kernel.
int pairwise_blocks_per_cu(int C, int K);
hipError_t launch_pairwise(int C, const EpochArgs& a, int grid, hipStream_t s);

}  // namespace w2v
