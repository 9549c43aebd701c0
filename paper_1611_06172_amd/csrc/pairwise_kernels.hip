// Algorithm 1 of the paper (the original word2vec Hogwild SGD, per pair) as
// a GPU epoch kernel on gfx950: the baseline HogBatch is measured against.
//
// Sentences, subsampling, windows and learning rates are those of the
// HogBatch epoch (sentence.h). What differs is the step: every input word i
// of a target runs its own K+1 logistic regressions, against the target
// (label 1) and K negatives of its own (label 0; draws 2 + iK + k of the
// target's stream, so input word 0 uses the HogBatch shared negatives; a
// draw equal to the target is skipped). Each pair's inner product uses the
// M_out row as moved by the pairs before it, that row moves right after its
// pair, and the M_in row of i moves once, after its K+1 pairs, by the sum of
// alpha * error * (M_out row as used).
//
// One wavefront per sentence. Per input word, up to kPairBlock output rows
// are gathered at once; since the M_in row is fixed during its K+1 pairs,
// all their inner products come from one transposing reduction, together
// with |a|^2. A later pair on a row already moved in the same block (a
// repeated negative) then sees x + (sum of earlier errors) |a|^2 and the
// row moved by those errors, exactly as if it had been re-read. Blocks and
// input words are processed in order; each gathers its rows after the
// previous one's writes were issued, so it reads them back moved. Update
// path as in HogBatch: fp32 atomics for ids < hot_rows, write-through
// stores otherwise.
#include "kernel_args.h"
#include "sentence.h"
#include "sgns_core.h"

namespace w2v {

constexpr int kPairBlock = 8;  // output rows gathered per reduction

// Negative k (lane k < K) of input word i of the target at raw position p.
__device__ __forceinline__ int pair_negative(const EpochArgs& a, int64_t p,
                                             int i, int k) {
  const int word = 2 + i * a.K + k;
  const U64x4 blk = stream_block(a.seed, (uint64_t)p, (uint64_t)a.epoch,
                                 (uint64_t)(word >> 3));
  const uint32_t r = word_of(blk, word & 7);
  return a.table[scale_draw(r, (uint64_t)a.table_size)];
}

template <int C>
__device__ __forceinline__ void write_row(float* M, int id, int64_t ld, int D,
                                          int lane, int hot_rows,
                                          const float (&old)[C],
                                          const float (&g)[C]) {
  update_row<C, false>(M, id, ld, D, lane, hot_rows, old, g);
}

template <int C>
__global__ __launch_bounds__(kWave) void k_epoch_pairwise(EpochArgs a) {
  __shared__ SentenceLds sl;
  __shared__ TargetBatch tb;
  extern __shared__ int32_t negs_lds[];  // [kWave][K], formed and unused
  const int lane = threadIdx.x;
  const int K = a.K;
  const int64_t ld = a.ld;
  const int D = a.D;
  const bool want_loss = a.loss != nullptr;

  int64_t n_mb = 0, sum_n = 0, raw = 0, rejected = 0, rows = 0;
  double lsum = 0.0, lcnt = 0.0;
  int bucket = -1;

  for (int64_t s = blockIdx.x; s < a.n_sent; s += gridDim.x) {
    const int64_t sb = a.pos_begin + s * a.L;
    const int64_t se = min(sb + (int64_t)a.L, a.pos_end);
    const int len = (int)(se - sb);
    raw += len;
    const int n_ret = keep_and_compact<false>(a, sb, len, lane, sl, rejected);

    for (int q0 = 0; q0 < n_ret; q0 += kWave) {
      form_targets<false>(a, sb, q0, n_ret, lane, sl, tb, negs_lds);
      const int cnt = min(kWave, n_ret - q0);
      for (int j = 0; j < cnt; ++j) {
        const int n = uniform_int(tb.n[j]);
        if (n == 0) continue;
        const int qj = q0 + j;
        const int64_t p = sb + sl.ret_off[qj];
        const int target = uniform_int(sl.ret_id[qj]);
        const int lo = uniform_int(tb.lo[j]);
        const float alpha = uniform_float(tb.alpha[j]);
        // Every private negative must be a row: otherwise skip the target.
        bool bad = false;
        for (int base = 0; base < n * K; base += kWave) {
          const int idx = base + lane;
          if (idx < n * K) {
            const int neg = pair_negative(a, p, idx / K, idx % K);
            bad |= (neg < 0 || neg >= a.V);
          }
        }
        if (__ballot(bad) != 0ull) {
          ++rejected;
          continue;
        }
        ++n_mb;
        sum_n += n;
        rows += (int64_t)n * (K + 2);  // per input word: its row, K + 1 output rows
        float loss_t = 0.f;  // lane-uniform

        for (int i = 0; i < n; ++i) {
          int jj = lo + i;
          if (jj >= qj) ++jj;
          const int cid = uniform_int(sl.ret_id[jj]);
          const int my_neg = lane < K ? pair_negative(a, p, i, lane) : -1;
          float av[C], temp[C];
          load_row<C, true>(a.M_in, cid, ld, D, lane, av);
#pragma unroll
          for (int c = 0; c < C; ++c) temp[c] = 0.f;

          for (int k0 = 0; k0 <= K; k0 += kPairBlock) {
            int ids[kPairBlock];
#pragma unroll
            for (int kk = 0; kk < kPairBlock; ++kk) {
              const int col = k0 + kk;
              int id = -1;
              if (col == 0) {
                id = target;
              } else if (col <= K) {
                id = __builtin_amdgcn_readlane(my_neg, col - 1);
                if (id == target) id = -1;  // masked: the pair is skipped
              }
              ids[kk] = id;
            }
            float o[kPairBlock][C];
#pragma unroll
            for (int kk = 0; kk < kPairBlock; ++kk) {
              if (ids[kk] >= 0) {
                load_row<C, true>(a.M_out, ids[kk], ld, D, lane, o[kk]);
              } else {
#pragma unroll
                for (int c = 0; c < C; ++c) o[kk][c] = 0.f;
              }
            }
            // Inner products of the block and |a|^2 in one reduction.
            float v[kWave];
#pragma unroll
            for (int kk = 0; kk < kPairBlock; ++kk) {
              float acc = 0.f;
#pragma unroll
              for (int c = 0; c < C; ++c) acc = fmaf(av[c], o[kk][c], acc);
              v[kk] = acc;
            }
            {
              float acc = 0.f;
#pragma unroll
              for (int c = 0; c < C; ++c) acc = fmaf(av[c], av[c], acc);
              v[kPairBlock] = acc;
            }
#pragma unroll
            for (int t = kPairBlock + 1; t < kWave; ++t) v[t] = 0.f;
            const float xs = xpose_reduce64(v, lane);
            const float aa = lane_value(xs, kPairBlock);

            // Pairs in order (lane-uniform): g = alpha (label - sigma(x)),
            // x taken after the earlier pairs of the block on the same row.
            float g[kPairBlock], before[kPairBlock];
#pragma unroll
            for (int kk = 0; kk < kPairBlock; ++kk) {
              g[kk] = 0.f;
              before[kk] = 0.f;
              if (ids[kk] < 0) continue;
              float prev = 0.f;
#pragma unroll
              for (int k2 = 0; k2 < kk; ++k2)
                if (ids[k2] == ids[kk]) prev += g[k2];
              const float x = lane_value(xs, kk) + prev * aa;
              const bool is_target = (k0 + kk == 0);
              const float z = is_target ? -x : x;
              const float sz = 1.f / (1.f + __expf(-z));
              g[kk] = alpha * (is_target ? sz : -sz);
              before[kk] = prev;
              if (want_loss) loss_t += softplus(z);
            }
            // temp += g * (row as used); each distinct row moves once by the
            // sum of its errors.
#pragma unroll
            for (int kk = 0; kk < kPairBlock; ++kk) {
              if (ids[kk] < 0) continue;
#pragma unroll
              for (int c = 0; c < C; ++c)
                temp[c] = fmaf(g[kk], fmaf(before[kk], av[c], o[kk][c]), temp[c]);
            }
#pragma unroll
            for (int kk = 0; kk < kPairBlock; ++kk) {
              if (ids[kk] < 0) continue;
              bool first = true;
              float total = g[kk];
#pragma unroll
              for (int k2 = 0; k2 < kPairBlock; ++k2) {
                if (k2 < kk && ids[k2] == ids[kk]) first = false;
                if (k2 > kk && ids[k2] == ids[kk]) total += g[k2];
              }
              if (!first) continue;
              float d[C];
#pragma unroll
              for (int c = 0; c < C; ++c) d[c] = total * av[c];
              write_row<C>(a.M_out, ids[kk], ld, D, lane, a.hot_rows, o[kk], d);
            }
          }
          write_row<C>(a.M_in, cid, ld, D, lane, a.hot_rows, av, temp);
        }

        if (want_loss) {
          const int b = (int)(p * (int64_t)a.n_buckets / a.T);
          if (b != bucket) {
            if (bucket >= 0) flush_loss(a.loss, bucket, lsum, lcnt, lane);
            bucket = b;
          }
          if (lane == 0) {
            lsum += (double)loss_t;
            lcnt += (double)n;
          }
        }
      }
      __syncthreads();
    }
  }
  if (want_loss && bucket >= 0) flush_loss(a.loss, bucket, lsum, lcnt, lane);
  flush_stats(a, lane, n_mb, sum_n, raw, rejected, rows);
}

// ------------------------------------------------------------ launchers --

using PairKernel = void (*)(EpochArgs);

static PairKernel pairwise_kernel_for(int C) {
  switch (C) {
    case 1: return k_epoch_pairwise<1>;
    case 2: return k_epoch_pairwise<2>;
    case 3: return k_epoch_pairwise<3>;
    case 4: return k_epoch_pairwise<4>;
    case 5: return k_epoch_pairwise<5>;
    case 6: return k_epoch_pairwise<6>;
    case 8: return k_epoch_pairwise<8>;
    case 10: return k_epoch_pairwise<10>;
    default: return nullptr;
  }
}

int pairwise_blocks_per_cu(int C, int K) {
  PairKernel k = pairwise_kernel_for(C);
  if (k == nullptr) return 0;
  const size_t dyn = sizeof(int32_t) * kWave * (size_t)(K > 0 ? K : 1);
  return resident_blocks_per_cu(reinterpret_cast<const void*>(k), dyn);
}

hipError_t launch_pairwise(int C, const EpochArgs& a, int grid, hipStream_t s) {
  PairKernel k = pairwise_kernel_for(C);
  if (k == nullptr) return hipErrorInvalidValue;
  const size_t dyn = sizeof(int32_t) * kWave * (size_t)(a.K > 0 ? a.K : 1);
  hipLaunchKernelGGL(k, dim3(grid), dim3(kWave), dyn, s, a);
  return hipGetLastError();
}

}  // namespace w2v
