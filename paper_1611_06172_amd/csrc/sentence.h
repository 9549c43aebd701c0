// Per-sentence minibatch formation on one wavefront (gfx950), shared by the
// epoch kernels and the minibatch export so that all of them draw the same
// minibatches.
//
//  * keep_and_compact: reads a sentence's raw ids, decides subsampling per
//    position (Philox word 0 against the keep threshold) and compacts the
//    kept words into LDS with a ballot prefix count.
//  * form_targets: forms up to 64 targets lane-parallel: window half-width
//    (word 1), the K shared negatives (words 2.., one table read each), the
//    decayed learning rate, and whether a negative id is out of range.
#pragma once

#include "device_common.h"
#include "kernel_args.h"

namespace w2v {

constexpr int kMaxSentence = 1024;
constexpr int kMaxWindow = 16;

struct SentenceLds {
  int32_t ret_id[kMaxSentence];   // kept word ids, in order
  int16_t ret_off[kMaxSentence];  // their offsets in the sentence
};

// Targets q0 .. q0+63 of a sentence.
struct TargetBatch {
  int32_t lo[kWave];              // first retained index of the window
  int32_t n[kWave];               // number of input words
  float alpha[kWave];
  uint64_t mask[kWave];           // bit k: negative k equals the target
  int32_t bad[kWave];             // a negative id outside [0, V)
};

__device__ __forceinline__ uint32_t word_of(const U64x4& b, int j) {
  const int m = j >> 1;
  const uint64_t v = m == 0 ? b.v[0] : m == 1 ? b.v[1] : m == 2 ? b.v[2] : b.v[3];
  return (j & 1) ? (uint32_t)(v >> 32) : (uint32_t)v;
}

// Subsampling and compaction of the sentence [sb, sb + len). Returns the
// number of kept words; counts out-of-range ids in `rejected`. The export
// variant marks every position that forms no minibatch with -1.
template <bool kExport>
__device__ __forceinline__ int keep_and_compact(const EpochArgs& a, int64_t sb,
                                                int len, int lane,
                                                SentenceLds& sl,
                                                int64_t& rejected) {
  const uint64_t e = (uint64_t)a.epoch;
  int n_ret = 0;
  for (int base = 0; base < len; base += kWave) {
    const int off = base + lane;
    const bool in = off < len;
    const int x = in ? a.corpus[sb + off] : 0;
    // -1 marks a word dropped from the vocabulary (w2v_build_vocab): it is
    // removed from the sentence before windows form, as any out-of-range id,
    // but it is no error.
    const bool bad = in && (x < -1 || x >= a.V);
    bool keep = in && x >= 0 && x < a.V;
    if (keep && a.thr != nullptr) {
      const U64x4 blk = stream_block(a.seed, (uint64_t)(sb + off), e, 0);
      keep = (uint32_t)blk.v[0] <= a.thr[x];
    }
    const uint64_t m = __ballot(keep);
    if (keep) {
      const int dst = n_ret + __popcll(m & lanes_below(lane));
      sl.ret_id[dst] = x;
      sl.ret_off[dst] = (int16_t)off;
    }
    n_ret += __popcll(m);
    rejected += __popcll(__ballot(bad));
    if (kExport && in && !keep) a.out_targets[sb + off - a.pos_begin] = -1;
  }
  __syncthreads();
  return n_ret;
}

// Forms targets q0 + lane (lane < n_batch <= 64, q0 + lane < n_ret) into tb
// and their negatives into negs[lane * K + k]. The export variant also
// writes the minibatches out.
template <bool kExport>
__device__ __forceinline__ void form_targets(const EpochArgs& a, int64_t sb,
                                             int q0, int n_ret, int lane,
                                             const SentenceLds& sl,
                                             TargetBatch& tb, int32_t* negs,
                                             int n_batch = kWave) {
  const uint64_t e = (uint64_t)a.epoch;
  const int K = a.K;
  const int w = a.w;
  const int q = q0 + lane;
  if (q < n_ret && lane < n_batch) {
    const int64_t p = sb + sl.ret_off[q];
    const int t = sl.ret_id[q];
    U64x4 blk = stream_block(a.seed, (uint64_t)p, e, 0);
    const int h = w - (int)scale_draw(word_of(blk, 1), (uint64_t)w);
    const int lo = max(q - h, 0);
    const int hi = min(q + h, n_ret - 1);
    const int n = hi - lo;
    uint64_t mask = 0;
    int bad = 0;
    int cur = 0;
    for (int k = 0; k < K; ++k) {
      const int word = 2 + k;
      if ((word >> 3) != cur) {
        cur = word >> 3;
        blk = stream_block(a.seed, (uint64_t)p, e, (uint64_t)cur);
      }
      const uint32_t r = word_of(blk, word & 7);
      const int neg = a.table[scale_draw(r, (uint64_t)a.table_size)];
      bad |= (neg < 0 || neg >= a.V);
      if (neg == t) mask |= 1ull << k;
      negs[lane * K + k] = neg;
    }
    const float alpha =
        decayed_alpha(a.alpha0, a.min_frac, a.epoch, a.n_epochs, a.T, p);
    tb.lo[lane] = lo;
    tb.n[lane] = n;
    tb.alpha[lane] = alpha;
    tb.mask[lane] = mask;
    tb.bad[lane] = bad;
    if constexpr (kExport) {
      const int64_t r = p - a.pos_begin;
      if (n == 0) {
        a.out_targets[r] = -1;
      } else {
        a.out_targets[r] = t;
        for (int i = 0; i < 2 * w; ++i) {
          int id = -1;
          if (i < n) id = sl.ret_id[lo + i + (lo + i >= q ? 1 : 0)];
          a.out_ctx[r * 2 * w + i] = id;
        }
        for (int k = 0; k < K; ++k) {
          a.out_negs[r * K + k] = negs[lane * K + k];
          a.out_mask[r * K + k] = (uint8_t)((mask >> k) & 1ull);
        }
        a.out_alpha[r] = alpha;
      }
    }
  }
  __syncthreads();
}

// Adds a wave's loss sums for one bucket (lane 0 holds the input count).
__device__ __forceinline__ void flush_loss(double* loss, int bucket,
                                           double& lsum, double& lcnt,
                                           int lane) {
  double s = lsum;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m);
  if (lane == 0) {
    unsafeAtomicAdd(loss + 2 * bucket, s);
    unsafeAtomicAdd(loss + 2 * bucket + 1, lcnt);
  }
  lsum = 0.0;
  lcnt = 0.0;
}

// Adds a wave's counters into stats[0..4] (lane 0) and raises the device's
// error word if the wave skipped anything for an id outside [0, V).
__device__ __forceinline__ void flush_stats(const EpochArgs& a, int lane,
                                            int64_t n_mb, int64_t sum_n,
                                            int64_t raw, int64_t rejected,
                                            int64_t rows) {
  int64_t* const stats = a.stats;
  if (lane == 0) report_bad_ids(a.status, rejected);
  if (stats != nullptr && lane == 0) {
    atomicAdd((unsigned long long*)&stats[0], (unsigned long long)n_mb);
    atomicAdd((unsigned long long*)&stats[1], (unsigned long long)sum_n);
    atomicAdd((unsigned long long*)&stats[2], (unsigned long long)raw);
    atomicAdd((unsigned long long*)&stats[3], (unsigned long long)rejected);
    atomicAdd((unsigned long long*)&stats[4], (unsigned long long)rows);
  }
}

}  // namespace w2v
