// Pipelined HogBatch epoch on gfx950 for shapes whose K+1 output columns fit
// one reduction block (the paper's K = 5 with windows up to 5).
//
// One wavefront owns one sentence at a time, as in the general kernel, and
// forms the same minibatches (sentence.h). What changes is how rows move:
//
//  * Input rows live in an LDS ring indexed by retained position: the window
//    of target q covers positions q-w..q+w, so consecutive targets share all
//    but one input row, and each step loads one entering row straight into
//    LDS (buffer load to LDS, no VGPRs). Updates to an input row are written
//    into the ring, so the wavefront sees its own updates at once. A row of
//    a rare word (id >= hot_rows) reaches M_in once, when it leaves the
//    window: its minibatch updates are summed in the ring first, the update
//    reduction of Sec. 1.1. A row of a frequent word is added to M_in
//    atomically every step and reloaded into the ring before every
//    minibatch that uses it, so it never goes stale for longer than the
//    general kernel would let it.
//  * Loads run one step ahead and each step has a single wait on global
//    memory, at its start: the output rows of q+1 and the entering row are
//    issued before minibatch q computes.
//  * Where a step's data overlaps the previous step's results the sequential
//    order is kept: an entering rare word already held in the ring is copied
//    from there, every ring slot holding an updated word receives the new
//    values, q+1's prefetched output rows take q's results for words both
//    use, and hot rows are reloaded after q's atomics. One wavefront
//    (max_inflight = 1) therefore reproduces the sequential epoch.
#include "kernel_args.h"
#include "sentence.h"
#include "sgns_core.h"

namespace w2v {

constexpr int kMaxRing = 2 * kMaxWindow + 2;

struct PipeLds {
  int ring_id[kMaxRing];     // word held by each ring slot, -1 = empty
  int raw_ctx[kMaxInputs];   // input words of the current minibatch
  int ctx_slot[kMaxInputs];  // ring slot of each distinct input word
  float cwgt[kMaxInputs];    // multiplicity of each distinct input word
  int raw_neg[kWave];
  int out[2][kWave];         // distinct output words, by minibatch parity
  float wgt[2][kWave];
  float E[kWave];
};

template <int C>
__device__ __forceinline__ void ring_read(const float* ring, int slot, int lane,
                                          float (&r)[C]) {
  const float* row = ring + slot * (C * kWave) + lane;
#pragma unroll
  for (int c = 0; c < C; ++c) r[c] = row[kWave * c];
}

template <int C>
__device__ __forceinline__ void ring_write(float* ring, int slot, int lane,
                                           const float (&r)[C]) {
  float* row = ring + slot * (C * kWave) + lane;
#pragma unroll
  for (int c = 0; c < C; ++c) row[kWave * c] = r[c];
}

template <int C>
__device__ __forceinline__ void store_row(float* M, int64_t id, int64_t ld,
                                          int D, int lane, const float (&r)[C]) {
  const __amdgpu_buffer_rsrc_t rs = row_rsrc(M + id * ld, D * 4);
#pragma unroll
  for (int c = 0; c < C; ++c)
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(r[c]), rs,
                                          (lane + kWave * c) * 4, 0, kPlainStore);
}

template <int C>
__device__ __forceinline__ void atomic_row(float* M, int64_t id, int64_t ld,
                                           int D, int lane, const float (&g)[C]) {
  const __amdgpu_buffer_rsrc_t rs = row_rsrc(M + id * ld, D * 4);
#pragma unroll
  for (int c = 0; c < C; ++c)
    __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(g[c], rs,
                                                    (lane + kWave * c) * 4, 0, 0);
}

// Stages the distinct output words of a minibatch (target first, masked and
// repeated negatives merged) into parity buffer par; returns their number.
__device__ __forceinline__ int stage_out(int lane, int target, int neg, int K,
                                         PipeLds& pl, int par) {
  if (lane < K) pl.raw_neg[lane] = neg;
  wave_sync();
  bool first = false;
  float mult = 0.f;
  if (lane < K && neg != target) {
    first = true;
    for (int k = 0; k < K; ++k) {
      if (pl.raw_neg[k] == neg) {
        if (k < lane) first = false;
        mult += 1.f;
      }
    }
  }
  const uint64_t m = __ballot(first);
  if (lane == 0) {
    pl.out[par][0] = target;
    pl.wgt[par][0] = 1.f;
  }
  if (first) {
    const int dst = 1 + __popcll(m & lanes_below(lane));
    pl.out[par][dst] = neg;
    pl.wgt[par][dst] = mult;
  }
  wave_sync();
  return 1 + __popcll(m);
}

// Loads one matrix row straight into LDS (one buffer load per 64 columns,
// lane l's word to slot[l + 64c]); columns past D read as 0 through the
// descriptor's range check.
template <int C>
__device__ __forceinline__ void dma_row(const float* M, int64_t id, int64_t ld,
                                        int D, int lane, float* slot) {
  const __amdgpu_buffer_rsrc_t rs = row_rsrc(M + id * ld, D * 4);
#pragma unroll
  for (int c = 0; c < C; ++c)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rs, (__attribute__((address_space(3))) void*)(slot + kWave * c), 4,
        (lane + kWave * c) * 4, 0, 0, kCoherentLoad);
}

template <int C, int NMAX>
__global__ __launch_bounds__(kWave) void k_epoch_pipe(EpochArgs a) {
  constexpr int KB = kWave / NMAX;
  constexpr int kSlots = NMAX * KB;
  constexpr int DP = C * kWave;  // ring slot length in floats
  __shared__ SentenceLds sl;
  __shared__ TargetBatch tb[2];
  __shared__ PipeLds pl;
  extern __shared__ int32_t dyn[];  // negatives [2][64][K], then the ring
  const int lane = threadIdx.x;
  const int K = a.K;
  const int w = a.w;
  const int R = 2 * w + 2;
  const int kpad = K > 0 ? K : 1;
  int32_t* negs = dyn;
  float* ring = (float*)(dyn + 2 * kWave * kpad);
  const bool want_loss = a.loss != nullptr;
  const int64_t ld = a.ld;
  const int D = a.D;
  const int hot = a.hot_rows;

  // Ring padding columns (>= D) must hold zeros: clear the ring once; every
  // later write to a padding column writes 0.
  for (int i = lane; i < R * DP; i += kWave) ring[i] = 0.f;
  wave_sync();

  int64_t n_mb = 0, sum_n = 0, raw = 0, rejected = 0;
  double lsum = 0.0, lcnt = 0.0;
  int bucket = -1;

  for (int64_t s = blockIdx.x; s < a.n_sent; s += gridDim.x) {
    const int64_t sb = a.pos_begin + s * a.L;
    const int64_t se = min(sb + (int64_t)a.L, a.pos_end);
    const int len = (int)(se - sb);
    raw += len;
    const int n_ret = keep_and_compact<false>(a, sb, len, lane, sl, rejected);
    if (n_ret < 2) continue;  // a single kept word forms no minibatch
    form_targets<false>(a, sb, 0, n_ret, lane, sl, tb[0], negs);
    if (n_ret > kWave)
      form_targets<false>(a, sb, kWave, n_ret, lane, sl, tb[1], negs + kWave * kpad);

    uint64_t dirty = 0;  // ring slots whose cold row holds unwritten updates

    // Ring slot lookup: the slot (other than `except`) holding word id, or -1.
    auto find_slot = [&](int id, int except) -> int {
      const int rid = lane < R ? pl.ring_id[lane] : -1;
      const uint64_t m = __ballot(lane < R && lane != except && rid == id);
      return m == 0ull ? -1 : (int)__builtin_ctzll(m);
    };

    // Position x takes its slot: a cold word already held elsewhere in the
    // ring is copied from there (that copy has this wavefront's updates);
    // otherwise the slot keeps what its load brought.
    auto enter = [&](int x) {
      const int id = uniform_int(sl.ret_id[x]);
      const int sx = x % R;
      if (id >= hot) {
        const int src = find_slot(id, sx);
        if (src >= 0) {
          float r[C];
          ring_read<C>(ring, src, lane, r);
          ring_write<C>(ring, sx, lane, r);
          dirty |= ((dirty >> src) & 1ull) << sx;
        }
      }
      if (lane == 0) pl.ring_id[sx] = id;
      wave_sync();
    };

    // Writes position e back to M_in if its slot holds unwritten updates.
    auto evict = [&](int e) {
      const int sx = e % R;
      if ((dirty >> sx) & 1ull) {
        float r[C];
        ring_read<C>(ring, sx, lane, r);
        store_row<C>(a.M_in, uniform_int(pl.ring_id[sx]), ld, D, lane, r);
        dirty &= ~(1ull << sx);
      }
      if (lane == 0) pl.ring_id[sx] = -1;
      wave_sync();
    };

    // Issues the load of position x into its (free) slot, unless its word is
    // hot (refreshed before use) or a cold copy is already in the ring.
    auto fetch = [&](int x) {
      const int id = uniform_int(sl.ret_id[x]);
      if (id < hot || find_slot(id, -1) >= 0) return;
      dma_row<C>(a.M_in, id, ld, D, lane, ring + (x % R) * DP);
    };

    // Input words of target q, first occurrence per word: lane i < n holds
    // its position; returns the ballot of first occurrences.
    auto inputs_of = [&](int q, int lo, int n, int& my_pos, int& my_id,
                         float& mult) -> uint64_t {
      my_pos = -1;
      my_id = -1;
      if (lane < n) {
        my_pos = lo + lane + (lo + lane >= q ? 1 : 0);
        my_id = sl.ret_id[my_pos];
        pl.raw_ctx[lane] = my_id;
      }
      wave_sync();
      bool first = false;
      mult = 0.f;
      if (lane < n) {
        first = true;
        for (int i = 0; i < n; ++i) {
          if (pl.raw_ctx[i] == my_id) {
            if (i < lane) first = false;
            mult += 1.f;
          }
        }
      }
      wave_sync();
      return __ballot(first);
    };

    // Prologue: positions 0..min(w, n_ret-1), all loaded fresh.
    if (lane < kMaxRing) pl.ring_id[lane] = -1;
    wave_sync();
    for (int x = 0; x <= min(w, n_ret - 1); ++x) {
      dma_row<C>(a.M_in, uniform_int(sl.ret_id[x]), ld, D, lane, ring + (x % R) * DP);
      if (lane == 0) pl.ring_id[x % R] = sl.ret_id[x];
    }
    wait_global();
    wave_sync();

    // Output rows of target q into o; returns their number (0 when q forms
    // no minibatch).
    auto prep = [&](int q, float (&o)[KB][C]) -> int {
      int n_out = 0;
      if (q < n_ret) {
        const int b = (q >> 6) & 1;
        const int j = q & (kWave - 1);
        const int n = uniform_int(tb[b].n[j]);
        const int bad = uniform_int(tb[b].bad[j]);
        if (n > 0 && bad == 0) {
          const int neg = lane < K ? negs[b * kWave * kpad + j * K + lane] : 0;
          n_out = stage_out(lane, uniform_int(sl.ret_id[q]), neg, K, pl, q & 1);
        }
      }
#pragma unroll
      for (int kk = 0; kk < KB; ++kk) {
        if (kk < n_out) {
          load_row<C, true>(a.M_out, uniform_int(pl.out[q & 1][kk]), ld, D, lane,
                            o[kk]);
        } else {
#pragma unroll
          for (int c = 0; c < C; ++c) o[kk][c] = 0.f;
        }
      }
      return n_out;
    };

    // One step. It opens with the step's only wait on global memory: the
    // loads issued during the previous step had its whole compute to land.
    //  1. q's prefetched output rows take q-1's results where words coincide;
    //  2. ring upkeep: position q+w takes its slot, q-w-1 is written back,
    //     position q+1+w is loaded into the freed slot;
    //  3. q+1's output rows are loaded into the buffer that held q-1's;
    //  4. minibatch q from the ring and registers; updates go to the ring
    //     and to global memory (atomics for hot rows, stores for outputs);
    //  5. the hot input rows of q+1 are reloaded into the ring, after q's
    //     atomics, so that they carry every update issued so far.
    auto step = [&](int q, float (&o)[KB][C], int n_out,
                    float (&o_nxt)[KB][C], int n_prev) -> int {
      wait_global();
      wave_sync();
      if (n_out > 0 && n_prev > 0) {
        const int par = q & 1;
        const int ppar = par ^ 1;
        bool hit = false;
        if (lane < n_out) {
          const int id = pl.out[par][lane];
          for (int k = 0; k < n_prev; ++k) hit |= (pl.out[ppar][k] == id);
        }
        if (__ballot(hit) != 0ull) {
#pragma unroll
          for (int kn = 0; kn < KB; ++kn) {
            if (kn < n_out) {
              const int id = uniform_int(pl.out[par][kn]);
#pragma unroll
              for (int k = 0; k < KB; ++k) {
                if (k < n_prev && uniform_int(pl.out[ppar][k]) == id) {
#pragma unroll
                  for (int c = 0; c < C; ++c) o[kn][c] = o_nxt[k][c];
                }
              }
            }
          }
        }
      }
      if (q > 0 && (q & (kWave - 1)) == 0 && q + kWave < n_ret) {
        const int b = ((q >> 6) + 1) & 1;
        form_targets<false>(a, sb, q + kWave, n_ret, lane, sl, tb[b],
                            negs + b * kWave * kpad);
      }
      if (q >= 1) {
        if (q + w < n_ret) enter(q + w);
        if (q - w - 1 >= 0) evict(q - w - 1);
      }
      if (q + 1 + w < n_ret) fetch(q + 1 + w);
      const int n_nxt = prep(q + 1, o_nxt);

      const int b = (q >> 6) & 1;
      const int j = q & (kWave - 1);
      const int n = uniform_int(tb[b].n[j]);
      if (n > 0 && n_out == 0) ++rejected;  // a negative id out of range
      if (n > 0 && n_out > 0) {
        ++n_mb;
        sum_n += n;
        const int lo = uniform_int(tb[b].lo[j]);
        const float alpha = uniform_float(tb[b].alpha[j]);
        const int par = q & 1;

        // Distinct input words (representative ring slots), multiplicities.
        int my_pos, my_id;
        float mult;
        const uint64_t fm = inputs_of(q, lo, n, my_pos, my_id, mult);
        if ((fm >> lane) & 1ull) {
          const int dst = __popcll(fm & lanes_below(lane));
          pl.ctx_slot[dst] = my_pos % R;
          pl.cwgt[dst] = mult;
        }
        wave_sync();
        const int n_in = __popcll(fm);

        // Logit block: per-lane partials, then the transposing reduction.
        float v[kWave];
#pragma unroll
        for (int i = 0; i < NMAX; ++i) {
          if (i < n_in) {
            float ar[C];
            ring_read<C>(ring, uniform_int(pl.ctx_slot[i]), lane, ar);
#pragma unroll
            for (int kk = 0; kk < KB; ++kk) {
              float acc = 0.f;
#pragma unroll
              for (int c = 0; c < C; ++c) acc = fmaf(ar[c], o[kk][c], acc);
              v[i * KB + kk] = acc;
            }
          } else {
#pragma unroll
            for (int kk = 0; kk < KB; ++kk) v[i * KB + kk] = 0.f;
          }
        }
#pragma unroll
        for (int t = kSlots; t < kWave; ++t) v[t] = 0.f;
        const float x = xpose_reduce64(v, lane);

        const int li = lane / KB;
        const int lk = lane % KB;
        const bool valid = lane < kSlots && li < n_in && lk < n_out;
        const float wgt = valid ? pl.wgt[par][lk] * pl.cwgt[li] : 0.f;
        const float z = (lk == 0) ? -x : x;
        const float sz = 1.f / (1.f + __expf(-z));
        pl.E[lane] = valid ? wgt * alpha * ((lk == 0) ? sz : -sz) : 0.f;
        float loss_part = 0.f;
        if (want_loss && valid) loss_part = wgt * softplus(z);
        wave_sync();

        // Input rows: dO accumulates E^T A, each row takes its E O update.
        float go[KB][C];
#pragma unroll
        for (int kk = 0; kk < KB; ++kk)
#pragma unroll
          for (int c = 0; c < C; ++c) go[kk][c] = 0.f;
#pragma unroll
        for (int i = 0; i < NMAX; ++i) {
          if (i < n_in) {
            const int slot = uniform_int(pl.ctx_slot[i]);
            float ar[C], gi[C];
            ring_read<C>(ring, slot, lane, ar);
#pragma unroll
            for (int c = 0; c < C; ++c) gi[c] = 0.f;
#pragma unroll
            for (int kk = 0; kk < KB; ++kk) {
              const float e = pl.E[i * KB + kk];
#pragma unroll
              for (int c = 0; c < C; ++c) {
                go[kk][c] = fmaf(e, ar[c], go[kk][c]);
                gi[c] = fmaf(e, o[kk][c], gi[c]);
              }
            }
            float an[C];
#pragma unroll
            for (int c = 0; c < C; ++c) an[c] = ar[c] + gi[c];
            const int id = uniform_int(pl.ring_id[slot]);
            const int rid = lane < R ? pl.ring_id[lane] : -1;
            uint64_t mirrors = __ballot(lane < R && rid == id);
            const uint64_t all = mirrors;
            while (mirrors != 0ull) {
              const int dst = (int)__builtin_ctzll(mirrors);
              mirrors &= mirrors - 1;
              ring_write<C>(ring, dst, lane, an);
            }
            if (id < hot) {
              atomic_row<C>(a.M_in, id, ld, D, lane, gi);
            } else {
              dirty |= all;
            }
          }
        }

        // Output rows: new value o + dO (kept in o for the next step's patch).
#pragma unroll
        for (int kk = 0; kk < KB; ++kk) {
          if (kk < n_out) {
            const int id = uniform_int(pl.out[par][kk]);
#pragma unroll
            for (int c = 0; c < C; ++c) o[kk][c] += go[kk][c];
            if (id < hot) {
              atomic_row<C>(a.M_out, id, ld, D, lane, go[kk]);
            } else {
              store_row<C>(a.M_out, id, ld, D, lane, o[kk]);
            }
          }
        }

        if (want_loss) {
          const int64_t p = sb + sl.ret_off[q];
          const int bk = (int)(p * (int64_t)a.n_buckets / a.T);
          if (bk != bucket) {
            if (bucket >= 0) flush_loss(a.loss, bucket, lsum, lcnt, lane);
            bucket = bk;
          }
          lsum += (double)loss_part;
          if (lane == 0) lcnt += (double)n;
        }
      }

      // 5. Fresh copies of q+1's hot input rows, after q's atomics.
      if (q + 1 < n_ret && n_nxt > 0) {
        const int b1 = ((q + 1) >> 6) & 1;
        const int j1 = (q + 1) & (kWave - 1);
        int p1, id1;
        float m1;
        const uint64_t f1 = inputs_of(q + 1, uniform_int(tb[b1].lo[j1]),
                                      uniform_int(tb[b1].n[j1]), p1, id1, m1);
        uint64_t hm = __ballot(((f1 >> lane) & 1ull) && id1 < hot);
        while (hm != 0ull) {
          const int l = (int)__builtin_ctzll(hm);
          hm &= hm - 1;
          const int pos = __builtin_amdgcn_readlane(p1, l);
          const int id = __builtin_amdgcn_readlane(id1, l);
          dma_row<C>(a.M_in, id, ld, D, lane, ring + (pos % R) * DP);
        }
      }
      wave_sync();
      return n_nxt;
    };

    float oa[KB][C], ob[KB][C];
    int n_cur = prep(0, oa), n_prev = 0;
    for (int q = 0; q < n_ret; q += 2) {
      int n_next = step(q, oa, n_cur, ob, n_prev);
      n_prev = n_cur;
      n_cur = n_next;
      if (q + 1 < n_ret) {
        n_next = step(q + 1, ob, n_cur, oa, n_prev);
        n_prev = n_cur;
        n_cur = n_next;
      }
    }

    // Sentence end: write back every input row still holding updates.
    wait_global();
    wave_sync();
    for (int x = max(0, n_ret - 1 - w); x < n_ret; ++x) evict(x);
  }
  if (want_loss && bucket >= 0) flush_loss(a.loss, bucket, lsum, lcnt, lane);
  flush_stats(a.stats, lane, n_mb, sum_n, raw, rejected);
}

// ------------------------------------------------------------ launchers --

#define W2V_PIPE_SHAPES(X) \
  X(1, 10) X(2, 10) X(3, 10) X(4, 10) X(5, 10) X(6, 10) X(8, 10) X(10, 10) \
  X(1, 16) X(2, 16) X(3, 16) X(4, 16) X(5, 16) X(1, 32) X(2, 32)

using PipeKernel = void (*)(EpochArgs);

static PipeKernel pipe_kernel_for(int C, int nmax) {
#define W2V_PICK(c, n) \
  if (C == c && nmax == n) return k_epoch_pipe<c, n>;
  W2V_PIPE_SHAPES(W2V_PICK)
#undef W2V_PICK
  return nullptr;
}

bool pipe_applies(int C, int nmax, int K) {
  return K + 1 <= kWave / nmax && pipe_kernel_for(C, nmax) != nullptr;
}

size_t pipe_dyn_lds(int C, int window, int K) {
  const size_t kpad = K > 0 ? (size_t)K : 1;
  return sizeof(int32_t) * 2 * kWave * kpad +
         sizeof(float) * (size_t)(2 * window + 2) * (size_t)C * kWave;
}

int pipe_blocks_per_cu(int C, int nmax, int window, int K) {
  PipeKernel k = pipe_kernel_for(C, nmax);
  if (k == nullptr) return 0;
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &blocks, k, kWave, pipe_dyn_lds(C, window, K)) != hipSuccess)
    return 0;
  return blocks;
}

hipError_t launch_pipe(int C, int nmax, const EpochArgs& a, int grid,
                       hipStream_t s) {
  PipeKernel k = pipe_kernel_for(C, nmax);
  if (k == nullptr) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k, dim3(grid), dim3(kWave), pipe_dyn_lds(C, a.w, a.K), s,
                     a);
  return hipGetLastError();
}

}  // namespace w2v
