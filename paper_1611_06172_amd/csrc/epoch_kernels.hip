// Sentence-parallel HogBatch epoch on gfx950.
//
// One wavefront owns one sentence at a time (a persistent grid strides over
// the sentences of the range). For its sentence it
//   1. reads the raw ids, decides subsampling per position (Philox word 0
//      against the keep threshold) and compacts the kept words into LDS with a
//      ballot prefix count;
//   2. forms 64 targets at a time lane-parallel: window half-width (word 1),
//      the K shared negatives (words 2.., one table read each) and the
//      decayed learning rate;
//   3. runs those targets' minibatches in sentence order through the fused
//      minibatch (sgns_core.h), so every minibatch of a sentence sees the
//      updates of the ones before it, while minibatches of different
//      sentences interleave without locks (Hogwild, Sec. 1.1).
// The export variant stops after step 2 and writes the minibatches out.
#include "kernel_args.h"
#include "sgns_core.h"

namespace w2v {

constexpr int kMaxSentence = 1024;

struct SentenceLds {
  int32_t ret_id[kMaxSentence];   // kept word ids, in order
  int16_t ret_off[kMaxSentence];  // their offsets in the sentence
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

template <int C, int NMAX, bool kMulti, bool kExport>
__global__ __launch_bounds__(kWave) void k_epoch(EpochArgs a) {
  __shared__ SentenceLds sl;
  __shared__ MinibatchLds mb;
  extern __shared__ int32_t negs_lds[];  // [kWave][K]
  const int lane = threadIdx.x;
  const uint64_t e = (uint64_t)a.epoch;
  const int K = a.K;
  const int w = a.w;
  const bool want_loss = a.loss != nullptr;

  int64_t n_mb = 0, sum_n = 0, raw = 0, rejected = 0;
  double lsum = 0.0, lcnt = 0.0;
  int bucket = -1;

  for (int64_t s = blockIdx.x; s < a.n_sent; s += gridDim.x) {
    const int64_t sb = a.pos_begin + s * a.L;
    const int64_t se = min(sb + (int64_t)a.L, a.pos_end);
    const int len = (int)(se - sb);
    raw += len;

    // 1. subsampling and compaction
    int n_ret = 0;
    for (int base = 0; base < len; base += kWave) {
      const int off = base + lane;
      const bool in = off < len;
      const int x = in ? a.corpus[sb + off] : 0;
      const bool bad = in && (x < 0 || x >= a.V);
      bool keep = in && !bad;
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

    for (int q0 = 0; q0 < n_ret; q0 += kWave) {
      // 2. targets q0 .. q0+63, one per lane
      const int q = q0 + lane;
      if (q < n_ret) {
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
          negs_lds[lane * K + k] = neg;
        }
        const float alpha = decayed_alpha(a.alpha0, a.min_frac, a.epoch,
                                          a.n_epochs, a.T, p);
        sl.lo[lane] = lo;
        sl.n[lane] = n;
        sl.alpha[lane] = alpha;
        sl.mask[lane] = mask;
        sl.bad[lane] = bad;
        if constexpr (kExport) {
          const int64_t r = p - a.pos_begin;
          if (n == 0) {
            a.out_targets[r] = -1;
          } else {
            a.out_targets[r] = t;
            for (int i = 0; i < 2 * w; ++i) {
              int id = -1;
              if (i < n) {
                const int jj = lo + i + (lo + i >= q ? 1 : 0);
                id = sl.ret_id[jj];
              }
              a.out_ctx[r * 2 * w + i] = id;
            }
            for (int k = 0; k < K; ++k) {
              a.out_negs[r * K + k] = negs_lds[lane * K + k];
              a.out_mask[r * K + k] = (uint8_t)((mask >> k) & 1ull);
            }
            a.out_alpha[r] = alpha;
          }
        }
      }
      __syncthreads();
      const int cnt = min(kWave, n_ret - q0);
      for (int j = 0; j < cnt; ++j) {
        const int n = uniform_int(sl.n[j]);
        if (n == 0) continue;
        if (uniform_int(sl.bad[j]) != 0) {
          ++rejected;
          continue;
        }
        ++n_mb;
        sum_n += n;
        if constexpr (!kExport) {
          const int qj = q0 + j;
          const int lo = uniform_int(sl.lo[j]);
          int ctx_id = 0;
          if (lane < n) {
            int jj = lo + lane;
            if (jj >= qj) ++jj;
            ctx_id = sl.ret_id[jj];
          }
          const int n_in = stage_inputs(lane, ctx_id, lane < n, mb);
          const int neg = lane < K ? negs_lds[j * K + lane] : 0;
          const int n_out = stage_outputs(lane, sl.ret_id[qj], neg, K, mb);
          float loss_part = 0.f;
          run_minibatch<C, NMAX, kMulti, true, false>(
              a.M_in, a.M_out, a.M_in, a.M_out, a.ld, a.D, lane, n_in, n_out,
              uniform_float(sl.alpha[j]), a.hot_rows, mb, want_loss,
              loss_part);
          if (want_loss) {
            const int64_t p = sb + sl.ret_off[qj];
            const int b = (int)(p * (int64_t)a.n_buckets / a.T);
            if (b != bucket) {
              if (bucket >= 0) flush_loss(a.loss, bucket, lsum, lcnt, lane);
              bucket = b;
            }
            lsum += (double)loss_part;
            if (lane == 0) lcnt += (double)n;
          }
        }
      }
      __syncthreads();
    }
  }
  if (want_loss && bucket >= 0) flush_loss(a.loss, bucket, lsum, lcnt, lane);
  if (a.stats != nullptr && lane == 0) {
    atomicAdd((unsigned long long*)&a.stats[0], (unsigned long long)n_mb);
    atomicAdd((unsigned long long*)&a.stats[1], (unsigned long long)sum_n);
    atomicAdd((unsigned long long*)&a.stats[2], (unsigned long long)raw);
    atomicAdd((unsigned long long*)&a.stats[3], (unsigned long long)rejected);
  }
}

// ------------------------------------------------------------ launchers --

#define W2V_TRAIN_SHAPES(X) \
  X(1, 10) X(2, 10) X(3, 10) X(4, 10) X(5, 10) X(6, 10) X(8, 10) X(10, 10) \
  X(1, 16) X(2, 16) X(3, 16) X(4, 16) X(5, 16) X(1, 32) X(2, 32)

using EpochKernel = void (*)(EpochArgs);

// Kernel for C columns per lane, up to nmax input words, and K negatives:
// the single-block variant when the K+1 output columns fit one reduction.
static EpochKernel train_kernel_for(int C, int nmax, int K) {
  const bool multi = K + 1 > kWave / (nmax > 0 ? nmax : 1);
#define W2V_PICK(c, n) \
  if (C == c && nmax == n) \
    return multi ? k_epoch<c, n, true, false> : k_epoch<c, n, false, false>;
  W2V_TRAIN_SHAPES(W2V_PICK)
#undef W2V_PICK
  return nullptr;
}

bool train_shape_supported(int C, int nmax) {
  return train_kernel_for(C, nmax, 0) != nullptr;
}

int columns_for(int D) {
  static const int kCols[] = {1, 2, 3, 4, 5, 6, 8, 10};
  for (int c : kCols)
    if (D <= kWave * c) return c;
  return 0;
}

int inputs_cap_for(int n) {
  if (n <= 10) return 10;
  if (n <= 16) return 16;
  if (n <= 32) return 32;
  return 0;
}

static size_t epoch_dyn_lds(const EpochArgs& a) {
  return sizeof(int32_t) * (size_t)kWave * (size_t)(a.K > 0 ? a.K : 1);
}

int train_blocks_per_cu(int C, int nmax, int K) {
  EpochKernel k = train_kernel_for(C, nmax, K);
  if (k == nullptr) return 0;
  int blocks = 0;
  const size_t dyn = sizeof(int32_t) * kWave * (size_t)(K > 0 ? K : 1);
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k, kWave, dyn) !=
      hipSuccess)
    return 0;
  return blocks;
}

hipError_t launch_train(int C, int nmax, const EpochArgs& a, int grid,
                        hipStream_t s) {
  EpochKernel k = train_kernel_for(C, nmax, a.K);
  if (k == nullptr) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k, dim3(grid), dim3(kWave), epoch_dyn_lds(a), s, a);
  return hipGetLastError();
}

hipError_t launch_export(const EpochArgs& a, int grid, hipStream_t s) {
  hipLaunchKernelGGL((k_epoch<1, 10, false, true>), dim3(grid), dim3(kWave),
                     epoch_dyn_lds(a), s, a);
  return hipGetLastError();
}

}  // namespace w2v
