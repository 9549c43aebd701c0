// The fused HogBatch minibatch on one wavefront (gfx950, wave64).
//
// One minibatch = N input words (rows of M_in) and the target plus K shared
// negatives (rows of M_out) (Sec. 1.1, negative sample sharing; Fig. 1
// right). The N x (K+1) logit block, the sigmoid error of Alg. 1 and both
// gradient products are formed here from rows gathered once:
//
//   X = A O^T   E = alpha (l - sigma(X))   dA = E O   dO = E^T A
//
// Rows are staged deduplicated. A negative equal to the target is masked;
// repeated negatives collapse into one column of weight m, and repeated input
// words into one row of weight m (m identical rows or columns have identical
// logits and errors, so one copy with its error scaled by m yields the same
// dA and dO). Every row is then read once and written once per minibatch:
// all reads precede the minibatch's own writes even when the output columns
// take several blocks, and a plain read-modify-write of a row cannot lose a
// sibling update from the same minibatch.
//
// Layout: lane l holds columns l, l+64, ..., l+64(C-1) of every gathered row
// in VGPRs (C = ceil(D/64) rounded up to a compiled size), loaded through
// range-checked buffer descriptors. Each (input word, output word) pair
// leaves a per-lane partial dot product; the wave-wide transposing reduction
// turns up to 64 such partials into one total per lane, the error is
// evaluated lane-parallel and read back per slot with v_readlane, and the
// two gradient products are lane-local FMAs.
//
// Update path (live matrices, RowTiers): rows with id < hot_rows receive
// fp32 atomic adds (frequent words, whose concurrent updates would otherwise
// overwrite each other), all other rows a store of (value read + update)
// written through to device scope, the Hogwild write the paper's threads
// perform (Sec. 1.1). Rows below
// split_rows (the head of the Zipf law, written by nearly every concurrent
// wavefront) are spread over kSplitParts partial rows: a wavefront adds its
// update atomically to the partial row of its group (blockIdx mod
// kSplitParts, i.e. its XCD under round-robin dispatch), and reads return
// the matrix row plus every partial row, so atomics to one address come from
// one XCD only and nothing is hidden from a reader. Snapshot batches add
// their updates with fp64 atomics into a delta buffer instead, or write them
// to staging rows for a sorted reduction (StagedRows).
//
// Pending input-row updates (PendingRows): consecutive targets of a
// sentence share most of their input words, so a training wavefront adds
// the updates of a cold input row to an LDS slot instead of the matrix, reads
// the row as (matrix row + its pending updates) while the word stays in the
// window, and adds the slot to the matrix once, atomically, when it lets
// the word go. The row traffic of the minibatch path is dominated by its
// writes; this turns about 2 window writes of an input row into one.
//
// Output columns are processed in blocks of KB = 64 / NMAX so that one
// block's partials fill one reduction; with K+1 <= KB (the paper's K = 5 with
// up to ten input words) the whole minibatch is a single block, compiled
// without the cross-block accumulation of the input-row updates.
#pragma once

#include "device_common.h"
#include "w2v.h"

namespace w2v {

constexpr int kMaxInputs = 32;   // input words per minibatch (2 * max window)
constexpr int kMaxOutputs = 65;  // target + up to 64 negatives
constexpr int kSplitParts = W2V_SPLIT_PARTS;

// Per-wavefront LDS staging of one minibatch's ids and multiplicities.
struct MinibatchLds {
  int raw_ctx[kMaxInputs];  // input words as formed
  int ctx[kMaxInputs];      // distinct input words (rows of M_in)
  float cwgt[kMaxInputs];   // multiplicity of each input row
  int raw[kWave];           // negatives as drawn
  int out[kMaxOutputs];     // [0] target, then distinct unmasked negatives
  float wgt[kMaxOutputs];   // multiplicity of each output column
  int slot[kMaxInputs];     // pending-update slot of each input row (PendingRows)
};

// Stages the input rows: the lanes with `present` set hold the input words
// in order. Returns the number of distinct input rows.
__device__ __forceinline__ int stage_inputs(int lane, int id, bool present,
                                            MinibatchLds& mb) {
  const uint64_t pm = __ballot(present);
  const int n_raw = __popcll(pm);
  if (present) mb.raw_ctx[__popcll(pm & lanes_below(lane))] = id;
  __syncthreads();
  bool first = false;
  float mult = 0.f;
  const int mine = lane < n_raw ? mb.raw_ctx[lane] : -1;
  if (lane < n_raw) {
    first = true;
    for (int i = 0; i < n_raw; ++i) {
      if (mb.raw_ctx[i] == mine) {
        if (i < lane) first = false;
        mult += 1.f;
      }
    }
  }
  const uint64_t m = __ballot(first);
  if (first) {
    const int dst = __popcll(m & lanes_below(lane));
    mb.ctx[dst] = mine;
    mb.cwgt[dst] = mult;
  }
  __syncthreads();
  return __popcll(m);
}

// Stages the output columns; `neg` is lane k's negative for k < K.
// Returns the number of distinct output columns (target included).
__device__ __forceinline__ int stage_outputs(int lane, int target, int neg,
                                             int K, MinibatchLds& mb) {
  if (lane < K) mb.raw[lane] = neg;
  __syncthreads();
  bool first = false;
  float mult = 0.f;
  if (lane < K && neg != target) {
    first = true;
    for (int k = 0; k < K; ++k) {
      if (mb.raw[k] == neg) {
        if (k < lane) first = false;
        mult += 1.f;
      }
    }
  }
  const uint64_t m = __ballot(first);
  if (lane == 0) {
    mb.out[0] = target;
    mb.wgt[0] = 1.f;
  }
  if (first) {
    const int dst = 1 + __popcll(m & lanes_below(lane));
    mb.out[dst] = neg;
    mb.wgt[dst] = mult;
  }
  __syncthreads();
  return 1 + __popcll(m);
}

// Raw buffer descriptor of one matrix row of n_bytes: loads past the end
// return 0 and stores/atomics past it are dropped by the hardware range
// check, so a row of D floats needs no per-lane bounds test.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const void* row,
                                                          int n_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(row), (short)0,
                                           n_bytes, kBufferWord3);
}

// Loads columns lane + 64c, c < C, of one row (0 past D).
template <int C, bool kLive>
__device__ __forceinline__ void load_row(const float* base, int64_t id,
                                         int64_t ld, int D, int lane,
                                         float (&r)[C]) {
  const __amdgpu_buffer_rsrc_t rs = row_rsrc(base + id * ld, D * 4);
#pragma unroll
  for (int c = 0; c < C; ++c)
    r[c] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
        rs, (lane + kWave * c) * 4, 0, kLive ? kCoherentLoad : 0));
}

// Applies update g to one row whose values as read are `old`: fp64 atomics
// into a delta buffer (kAccum64), fp32 atomics for hot rows, otherwise a
// plain store of old + g.
template <int C, bool kAccum64>
__device__ __forceinline__ void update_row(void* base, int64_t id, int64_t ld,
                                           int D, int lane, int hot_rows,
                                           const float (&old)[C],
                                           const float (&g)[C]) {
  if constexpr (kAccum64) {
    double* row = (double*)base + id * ld;
#pragma unroll
    for (int c = 0; c < C; ++c)
      if (lane + kWave * c < D) unsafeAtomicAdd(row + lane + kWave * c, (double)g[c]);
  } else {
    const __amdgpu_buffer_rsrc_t rs = row_rsrc((float*)base + id * ld, D * 4);
    if (id < hot_rows) {
#pragma unroll
      for (int c = 0; c < C; ++c)
        __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(
            g[c], rs, (lane + kWave * c) * 4, 0, 0);
    } else {
#pragma unroll
      for (int c = 0; c < C; ++c)
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(old[c] + g[c]), rs,
                                              (lane + kWave * c) * 4, 0,
                                              kCoherentStore);
    }
  }
}

// log(1 + e^z) = -log sigma(-z), without overflow.
__device__ __forceinline__ float softplus(float z) {
  return fmaxf(z, 0.f) + log1pf(__expf(-fabsf(z)));
}

// Row access of a minibatch's live rows by tier: rows id < split_rows of
// matrix m (0: input, 1: output) have partial rows part[((m split_rows + id)
// kSplitParts + g) ld], g < kSplitParts, that every read adds and that take
// the updates (atomically, in the partial row of this wavefront's group);
// rows id < hot_rows take fp32 atomic adds; other rows a store of old + g.
// kAccum64: fp64 atomic adds into a delta buffer instead (snapshot batches).
template <int C, bool kAccum64>
struct RowTiers {
  float* part;
  int split_rows;
  int hot_rows;
  int64_t ld;
  int D;
  int lane;

  __device__ __forceinline__ float* part_base(int m, int id) const {
    return part + (int64_t)(m * split_rows + id) * kSplitParts * ld;
  }
  // Adds the partial rows of a split row to its value as read.
  __device__ __forceinline__ void add_split(int m, int id, float (&r)[C]) const {
    if (id < split_rows) {
      float* pb = part_base(m, id);
#pragma unroll 1
      for (int g = 0; g < kSplitParts; ++g) {
        float t[C];
        load_row<C, true>(pb, g, ld, D, lane, t);
#pragma unroll
        for (int c = 0; c < C; ++c) r[c] += t[c];
      }
    }
  }
  // Adds g to row id atomically whatever its tier (pending updates).
  __device__ __forceinline__ void add(int m, float* W, int id,
                                      const float (&g)[C]) const {
    if (id < split_rows)
      update_row<C, false>(part_base(m, id), blockIdx.x % kSplitParts, ld, D,
                           lane, kSplitParts, g, g);
    else
      update_row<C, false>(W, id, ld, D, lane, id + 1, g, g);
  }
  __device__ __forceinline__ void update(int m, void* W, int id,
                                         const float (&old)[C],
                                         const float (&g)[C]) const {
    if (id < split_rows) {
      update_row<C, false>(part_base(m, id), blockIdx.x % kSplitParts, ld, D,
                           lane, kSplitParts, old, g);
    } else {
      update_row<C, kAccum64>(W, id, ld, D, lane, hot_rows, old, g);
    }
  }
};

// Error and loss of slot (input row li, output column lk) of a minibatch of
// one target: column 0 is the target (label 1), the others negatives
// (label 0); both scaled by the row and column multiplicities.
struct TargetError {
  __device__ __forceinline__ float operator()(const MinibatchLds& mb, int li,
                                              int lk, float x, float alpha,
                                              bool want_loss,
                                              float& loss_part) const {
    const float wgt = mb.wgt[lk] * mb.cwgt[li];
    // label - sigma(x) is sigma(-x) for the target and -sigma(x) for a
    // negative; evaluating sigma(z) directly avoids cancelling against 1.
    const float z = (lk == 0) ? -x : x;
    const float sz = 1.f / (1.f + __expf(-z));
    if (want_loss) loss_part += wgt * softplus(z);
    return wgt * alpha * ((lk == 0) ? sz : -sz);
  }
};

// Input-row updates applied to the matrix at once (no pending slots).
struct NoPendingRows {
  template <int C>
  __device__ __forceinline__ void add_pending(int, int, float (&)[C]) const {}
  template <int C>
  __device__ __forceinline__ bool defer(int, int, const float (&)[C]) const {
    return false;
  }
  template <int C>
  __device__ __forceinline__ bool defer_out(int, int, const float (&)[C]) const {
    return false;
  }
};

// rows: [slots][64 C] floats in LDS, the updates a wavefront has made to an
// input row and not yet added to the matrix (lane l's columns l + 64c at
// offset 64c + l). slot[i] for distinct input i of the minibatch: -1: no
// slot, its update goes to the matrix at once; s < kSlotHeld: slot s,
// empty, which takes this minibatch's update; kSlotHeld + s: slot s holds
// pending updates of this word, which every read adds and to which this
// minibatch's update is added.
constexpr int kSlotHeld = 64;

struct PendingRows {
  float* rows;
  const int* slot;

  template <int C>
  __device__ __forceinline__ void add_pending(int i, int lane,
                                              float (&r)[C]) const {
    const int s = uniform_int(slot[i]);
    if (s < kSlotHeld) return;
    const float* p = rows + (s - kSlotHeld) * (kWave * C) + lane;
#pragma unroll
    for (int c = 0; c < C; ++c) r[c] += p[kWave * c];
  }
  template <int C>
  __device__ __forceinline__ bool defer(int i, int lane,
                                        const float (&g)[C]) const {
    const int s = uniform_int(slot[i]);
    if (s < 0) return false;
    float* p = rows + (s & (kSlotHeld - 1)) * (kWave * C) + lane;
    if (s >= kSlotHeld) {
#pragma unroll
      for (int c = 0; c < C; ++c) p[kWave * c] += g[c];
    } else {
#pragma unroll
      for (int c = 0; c < C; ++c) p[kWave * c] = g[c];
    }
    return true;
  }
  template <int C>
  __device__ __forceinline__ bool defer_out(int, int, const float (&)[C]) const {
    return false;
  }
};

// Updates written out instead of applied (sorted snapshot batches): the
// update of distinct input i goes to row i of `in`, that of output column k
// to row k of `out` (row stride ld; columns past D are not written).
struct StagedRows {
  float* in;
  float* out;
  int64_t ld;
  int D;

  template <int C>
  __device__ __forceinline__ void add_pending(int, int, float (&)[C]) const {}
  template <int C>
  __device__ __forceinline__ void put(float* row, int lane,
                                      const float (&g)[C]) const {
#pragma unroll
    for (int c = 0; c < C; ++c)
      if (lane + kWave * c < D) row[lane + kWave * c] = g[c];
  }
  template <int C>
  __device__ __forceinline__ bool defer(int i, int lane, const float (&g)[C]) const {
    put<C>(in + i * ld, lane, g);
    return true;
  }
  template <int C>
  __device__ __forceinline__ bool defer_out(int k, int lane,
                                            const float (&g)[C]) const {
    put<C>(out + k * ld, lane, g);
    return true;
  }
};

// Runs one minibatch. Rin/Rout: where rows are read; Win/Wout: where updates
// go (the same fp32 matrices, or fp64 delta buffers with the same row stride
// when kAccum64). n distinct input rows (n <= NMAX) in mb.ctx/mb.cwgt, n_out
// distinct output columns in mb.out/mb.wgt. Rows id < split_rows of matrix m
// (0: input, 1: output) have partial rows part[((m split_rows + id)
// kSplitParts + g) ld], g < kSplitParts (live matrices only). `err` gives
// the error of a slot (TargetError for one target); `pend` may take updates
// instead of the matrices: pending input rows (PendingRows), staging rows
// (StagedRows), or none (NoPendingRows).
// Every lane returns its share of the minibatch loss in `loss_part` when
// want_loss is set.
template <int C, int NMAX, bool kMulti, bool kLiveRead, bool kAccum64,
          class Err = TargetError, class Pend = NoPendingRows>
__device__ __forceinline__ void run_minibatch(
    const float* Rin, const float* Rout, void* Win, void* Wout, int64_t ld,
    int D, int lane, int n, int n_out, float alpha, int hot_rows,
    MinibatchLds& mb, bool want_loss, float& loss_part,
    float* part = nullptr, int split_rows = 0, const Err& err = Err(),
    const Pend& pend = Pend()) {
  const RowTiers<C, kAccum64> io{part, split_rows, hot_rows, ld, D, lane};
  auto read_split = [&](int m, int id, float (&r)[C]) { io.add_split(m, id, r); };
  auto update = [&](int m, void* W, int id, const float (&old)[C],
                    const float (&g)[C]) { io.update(m, W, id, old, g); };
  constexpr int KB = kWave / NMAX;
  constexpr int kSlots = NMAX * KB;
  static_assert(KB >= 1 && kSlots <= kWave, "NMAX must be <= 64");

  // Gather the input-word rows once (rows >= n stay zero).
  float a[NMAX][C];
#pragma unroll
  for (int i = 0; i < NMAX; ++i) {
    if (i < n) {
      load_row<C, kLiveRead>(Rin, uniform_int(mb.ctx[i]), ld, D, lane, a[i]);
      read_split(0, uniform_int(mb.ctx[i]), a[i]);
      pend.template add_pending<C>(i, lane, a[i]);
    } else {
#pragma unroll
      for (int c = 0; c < C; ++c) a[i][c] = 0.f;
    }
  }
  // Input-row updates accumulate over output blocks (kMulti); with a single
  // block (n_out <= KB guaranteed by the caller) they are applied directly.
  float ga[kMulti ? NMAX : 1][C];
  if constexpr (kMulti) {
#pragma unroll
    for (int i = 0; i < NMAX; ++i)
#pragma unroll
      for (int c = 0; c < C; ++c) ga[i][c] = 0.f;
  }

  // Output rows of the block starting at column k0 (zero past n_out).
  auto load_block = [&](int k0, float (&o)[KB][C]) {
#pragma unroll
    for (int kk = 0; kk < KB; ++kk) {
      if (k0 + kk < n_out) {
        load_row<C, kLiveRead>(Rout, uniform_int(mb.out[k0 + kk]), ld, D, lane,
                               o[kk]);
        read_split(1, uniform_int(mb.out[k0 + kk]), o[kk]);
      } else {
#pragma unroll
        for (int c = 0; c < C; ++c) o[kk][c] = 0.f;
      }
    }
  };
  // With several blocks, the next block's rows are loaded while this one is
  // computed and written; they are other rows than this block's (columns
  // are distinct), so every row is still read before the minibatch writes
  // it. The KB x C extra registers cost the C = 5, KB = 6 kernel its second
  // wavefront per SIMD (1e8 tokens, D = 300, K = 15: 123 -> 91 Mwords/s),
  // so it keeps the serial loads; the others gain (D = 100, K = 15: 144 ->
  // 180; D = 600, K = 15: 54 -> 63).
  constexpr bool kPrefetch = kMulti && (C * KB <= 24 || C >= 6);
  float next[kPrefetch ? KB : 1][C];
  if constexpr (kPrefetch) load_block(0, next);

  for (int k0 = 0; k0 < (kMulti ? n_out : 1); k0 += KB) {
    float o[KB][C];
    if constexpr (kPrefetch) {
#pragma unroll
      for (int kk = 0; kk < KB; ++kk)
#pragma unroll
        for (int c = 0; c < C; ++c) o[kk][c] = next[kk][c];
      if (k0 + KB < n_out) load_block(k0 + KB, next);
    } else {
      load_block(k0, o);
    }

    // Per-lane partial logits, slot s = i*KB + kk, formed as the reduction
    // consumes them.
    auto partial = [&](int s) -> float {
      const int i = s / KB;
      const int kk = s % KB;
      if (s >= kSlots || i >= n) return 0.f;
      float acc = 0.f;
#pragma unroll
      for (int c = 0; c < C; ++c) acc = fmaf(a[i][c], o[kk][c], acc);
      return acc;
    };
    const float x = xpose_reduce64_lazy(partial, lane);

    // Error of slot `lane` (input row li, output column lk).
    const int li = lane / KB;
    const int lk = k0 + lane % KB;
    const bool valid = lane < kSlots && li < n && lk < n_out;
    // Lane s keeps the error of slot s; the gradient products read it back
    // with v_readlane (a scalar operand of the FMAs, no LDS round trip).
    float e_lane = 0.f;
    if (valid) e_lane = err(mb, li, lk, x, alpha, want_loss, loss_part);

    // dO = E^T A for the block's output rows.
#pragma unroll
    for (int kk = 0; kk < KB; ++kk) {
      const int k = k0 + kk;
      if (k < n_out) {
        float g[C];
#pragma unroll
        for (int c = 0; c < C; ++c) g[c] = 0.f;
#pragma unroll
        for (int i = 0; i < NMAX; ++i) {
          if (i < n) {
            const float e = lane_value(e_lane, i * KB + kk);
#pragma unroll
            for (int c = 0; c < C; ++c) g[c] = fmaf(e, a[i][c], g[c]);
          }
        }
        if (!pend.template defer_out<C>(k, lane, g))
          update(1, Wout, uniform_int(mb.out[k]), o[kk], g);
      }
    }

    // dA = E O (accumulated over output blocks when there are several).
#pragma unroll
    for (int i = 0; i < NMAX; ++i) {
      if (i < n) {
        float g[C];
#pragma unroll
        for (int c = 0; c < C; ++c) g[c] = kMulti ? ga[kMulti ? i : 0][c] : 0.f;
#pragma unroll
        for (int kk = 0; kk < KB; ++kk) {
          const float e = lane_value(e_lane, i * KB + kk);
#pragma unroll
          for (int c = 0; c < C; ++c) g[c] = fmaf(e, o[kk][c], g[c]);
        }
        if constexpr (kMulti) {
#pragma unroll
          for (int c = 0; c < C; ++c) ga[i][c] = g[c];
        } else {
          if (!pend.template defer<C>(i, lane, g))
            update(0, Win, uniform_int(mb.ctx[i]), a[i], g);
        }
      }
    }
    __syncthreads();
  }
  if constexpr (kMulti) {
#pragma unroll
    for (int i = 0; i < NMAX; ++i)
      if (i < n) {
        if (!pend.template defer<C>(i, lane, ga[i]))
          update(0, Win, uniform_int(mb.ctx[i]), a[i], ga[i]);
      }
  }
}

}  // namespace w2v
