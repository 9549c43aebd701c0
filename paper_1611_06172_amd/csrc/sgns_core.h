// The fused HogBatch minibatch on one wavefront (gfx950, wave64).
//
// One minibatch = N input words (rows of M_in) and the target plus K shared
// negatives (rows of M_out) (Sec. 1.1, negative sample sharing; Fig. 1
// right). The N x (K+1) logit block, the sigmoid error of Alg. 1 and both
// gradient products are formed here from rows gathered once:
//
//   X = A O^T   E = alpha (l - sigma(X))   dA = E O   dO = E^T A
//
// Output columns are staged deduplicated: a negative equal to the target is
// masked (weight 0) and repeated negatives collapse into one column of
// weight m (m identical columns have identical rows, logits and errors, so
// one column with its error scaled by m gives the same dA and dO). Every
// output row is then read at most once per minibatch, which keeps all of a
// minibatch's reads ahead of its own writes even when the columns are
// processed in several blocks.
//
// Layout: lane l holds columns l, l+64, ..., l+64(C-1) of every gathered row
// in VGPRs (C = ceil(D/64) rounded up to a compiled size). Each (input word,
// output word) pair leaves a per-lane partial dot product; the wave-wide
// transposing reduction turns up to 64 such partials into one total per lane,
// the error is evaluated lane-parallel and broadcast through LDS, and the two
// gradient products are lane-local FMAs. Updates leave as one 64-wide
// coalesced atomic add per row and column block: fp32 adds into the live
// matrices (epoch training) or fp64 adds into a delta buffer (snapshot
// batches, rounded once per element afterwards).
//
// Output columns are processed in blocks of KB = 64 / NMAX so that one
// block's partials fill one reduction; with K+1 <= KB (the paper's K = 5 with
// up to ten input words) the whole minibatch is a single block.
#pragma once

#include "device_common.h"

namespace w2v {

constexpr int kMaxInputs = 32;   // input words per minibatch (2 * max window)
constexpr int kMaxOutputs = 65;  // target + up to 64 negatives

// Per-wavefront LDS staging of one minibatch's ids and its error block.
struct MinibatchLds {
  int ctx[kMaxInputs];      // input word ids (rows of M_in)
  int raw[kWave];           // negatives as drawn
  int out[kMaxOutputs];     // [0] target, then distinct unmasked negatives
  float wgt[kMaxOutputs];   // multiplicity of each output column
  float E[kWave];           // error block of the current output block
};

// Stages the output columns of a minibatch; `neg` is lane k's negative for
// k < K. Returns the number of distinct output columns (target included).
__device__ __forceinline__ int stage_outputs(int lane, int target, int neg,
                                             int K, MinibatchLds& mb) {
  if (lane < K) mb.raw[lane] = neg;
  __syncthreads();
  bool first = false;
  float mult = 0.f;
  if (lane < K && neg != target) {
    first = true;
    for (int k = 0; k < K; ++k) {
      const int other = mb.raw[k];
      if (other == neg) {
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

template <bool kLive>
__device__ __forceinline__ float load_row_elem(const float* p) {
  if constexpr (kLive) {
    return load_live(p);
  } else {
    return *p;
  }
}

template <bool kAccum64>
__device__ __forceinline__ void add_update(void* base, int64_t off, float g) {
  if constexpr (kAccum64) {
    unsafeAtomicAdd((double*)base + off, (double)g);
  } else {
    add_live((float*)base + off, g);
  }
}

// log(1 + e^z) = -log sigma(-z), without overflow.
__device__ __forceinline__ float softplus(float z) {
  return fmaxf(z, 0.f) + log1pf(__expf(-fabsf(z)));
}

// Runs one minibatch. Rin/Rout: where rows are read; Win/Wout: where updates
// are added (fp32 matrices, or fp64 delta buffers with the same row stride
// when kAccum64). n input words (n <= NMAX) in mb.ctx, n_out staged output
// columns in mb.out/mb.wgt. Every lane returns its share of the minibatch
// loss in `loss_part` when want_loss is set.
template <int C, int NMAX, bool kLiveRead, bool kAccum64>
__device__ __forceinline__ void run_minibatch(
    const float* Rin, const float* Rout, void* Win, void* Wout, int64_t ld,
    int D, int lane, int n, int n_out, float alpha, MinibatchLds& mb,
    bool want_loss, float& loss_part) {
  constexpr int KB = kWave / NMAX;
  static_assert(KB >= 1, "NMAX must be <= 64");
  bool ok[C];
#pragma unroll
  for (int c = 0; c < C; ++c) ok[c] = lane + kWave * c < D;

  // Gather the input-word rows once.
  float a[NMAX][C];
#pragma unroll
  for (int i = 0; i < NMAX; ++i) {
    if (i < n) {
      const int id = uniform_int(mb.ctx[i]);
      const float* row = Rin + (int64_t)id * ld + lane;
#pragma unroll
      for (int c = 0; c < C; ++c)
        a[i][c] = ok[c] ? load_row_elem<kLiveRead>(row + kWave * c) : 0.f;
    } else {
#pragma unroll
      for (int c = 0; c < C; ++c) a[i][c] = 0.f;
    }
  }

  for (int k0 = 0; k0 < n_out; k0 += KB) {
    float o[KB][C];
#pragma unroll
    for (int kk = 0; kk < KB; ++kk) {
      if (k0 + kk < n_out) {
        const int id = uniform_int(mb.out[k0 + kk]);
        const float* row = Rout + (int64_t)id * ld + lane;
#pragma unroll
        for (int c = 0; c < C; ++c)
          o[kk][c] = ok[c] ? load_row_elem<kLiveRead>(row + kWave * c) : 0.f;
      } else {
#pragma unroll
        for (int c = 0; c < C; ++c) o[kk][c] = 0.f;
      }
    }

    // Per-lane partial logits of the block, slot i*KB + kk.
    float v[kWave];
#pragma unroll
    for (int i = 0; i < NMAX; ++i) {
#pragma unroll
      for (int kk = 0; kk < KB; ++kk) {
        float acc = 0.f;
        if (i < n) {
#pragma unroll
          for (int c = 0; c < C; ++c) acc = fmaf(a[i][c], o[kk][c], acc);
        }
        v[i * KB + kk] = acc;
      }
    }
#pragma unroll
    for (int s = NMAX * KB; s < kWave; ++s) v[s] = 0.f;
    const float x = xpose_reduce64(v, lane);

    // Error of slot `lane` (input li, output column lk).
    const int li = lane / KB;
    const int lk = k0 + lane % KB;
    const bool valid = lane < NMAX * KB && li < n && lk < n_out;
    const float wgt = valid ? mb.wgt[lk] : 0.f;
    // label - sigma(x) is sigma(-x) for the target and -sigma(x) for a
    // negative; evaluating sigma(z) directly avoids cancelling against 1.
    const float z = (lk == 0) ? -x : x;
    const float sz = 1.f / (1.f + __expf(-z));
    mb.E[lane] = valid ? wgt * alpha * ((lk == 0) ? sz : -sz) : 0.f;
    if (want_loss && valid) loss_part += wgt * softplus(z);
    __syncthreads();

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
            const float e = mb.E[i * KB + kk];
#pragma unroll
            for (int c = 0; c < C; ++c) g[c] = fmaf(e, a[i][c], g[c]);
          }
        }
        const int64_t off = (int64_t)uniform_int(mb.out[k]) * ld + lane;
#pragma unroll
        for (int c = 0; c < C; ++c)
          if (ok[c]) add_update<kAccum64>(Wout, off + kWave * c, g[c]);
      }
    }

    // dA = E O for every input row (per block when there are several).
#pragma unroll
    for (int i = 0; i < NMAX; ++i) {
      if (i < n) {
        float g[C];
#pragma unroll
        for (int c = 0; c < C; ++c) g[c] = 0.f;
#pragma unroll
        for (int kk = 0; kk < KB; ++kk) {
          const float e = mb.E[i * KB + kk];
#pragma unroll
          for (int c = 0; c < C; ++c) g[c] = fmaf(e, o[kk][c], g[c]);
        }
        const int64_t off = (int64_t)uniform_int(mb.ctx[i]) * ld + lane;
#pragma unroll
        for (int c = 0; c < C; ++c)
          if (ok[c]) add_update<kAccum64>(Win, off + kWave * c, g[c]);
      }
    }
    __syncthreads();
  }
}

}  // namespace w2v
