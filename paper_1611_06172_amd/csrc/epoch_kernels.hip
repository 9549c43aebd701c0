// Sentence-parallel HogBatch epoch on gfx950: the general kernel.
//
// One wavefront owns one sentence at a time (a persistent grid strides over
// the sentences of the range). For its sentence it
//   1. decides subsampling and compacts the kept words (sentence.h);
//   2. forms up to 64 targets at a time lane-parallel (sentence.h; fewer
//      where their negatives would cost LDS residency);
//   3. runs those targets' minibatches in sentence order through the fused
//      minibatch (sgns_core.h), so every minibatch of a sentence sees the
//      updates of the ones before it, while minibatches of different
//      sentences interleave without locks (Hogwild, Sec. 1.1). The updates
//      of cold input rows collect in a few LDS slots while their words stay
//      in the window (assign_slots, PendingRows) and reach the matrix once.
// It serves every compiled shape, including output blocks that take several
// reductions. The export variant stops after step 2 and writes the
// minibatches out.
#include <climits>
#include <map>
#include <mutex>
#include <tuple>

#include "group_core.h"
#include "kernel_args.h"
#include "sentence.h"
#include "sgns_core.h"

namespace w2v {

// Pending-update slots of a wavefront: lane s < nslots holds the word of
// slot s (slot_id, -1 if free) and the retained index of the last target
// that used it (slot_t). For the minibatch of target qj with distinct inputs
// mb.ctx[0..n):
//   * a word held in a slot is a hit;
//   * any other word with id >= pend_from takes a free slot, else the least
//     recently used slot no input of this minibatch holds (whose pending
//     updates flush(s, id) first adds to the matrix), else none (its update
//     goes to the matrix at once).
// The choice goes to mb.slot (PendingRows). Slots unused for more than
// `expire` targets are flushed and freed first, so no update stays pending
// after its word has left the window for good; the caller flushes every
// slot at the end of a sentence.
template <int NMAX, class Flush>
__device__ __forceinline__ void assign_slots(MinibatchLds& mb, int n, int qj,
                                             int expire, int nslots,
                                             int pend_from, int lane,
                                             int& slot_id, int& slot_t,
                                             const Flush& flush) {
  const bool mine = lane < nslots;
  for (uint64_t old = __ballot(mine && slot_id >= 0 && slot_t < qj - expire);
       old != 0ull; old &= old - 1ull) {
    const int s = __builtin_ctzll(old);
    flush(s, __builtin_amdgcn_readlane(slot_id, s));
    if (lane == s) slot_id = -1;
  }
  int code = -1;       // lane i < n: slot code of input i
  uint32_t done = 0u;  // inputs settled by the first pass
#pragma unroll
  for (int i = 0; i < NMAX; ++i) {
    if (i < n) {
      const int id = uniform_int(mb.ctx[i]);
      const uint64_t hm = __ballot(mine && slot_id == id);
      if (hm != 0ull || id < pend_from) done |= 1u << i;
      if (hm != 0ull) {
        const int s = __builtin_ctzll(hm);
        if (lane == i) code = kSlotHeld + s;
        if (lane == s) slot_t = qj;
      }
    }
  }
#pragma unroll
  for (int i = 0; i < NMAX; ++i) {
    if (i < n && ((done >> i) & 1u) == 0u) {
      const int key = !mine ? INT_MAX : slot_id < 0 ? -1 : slot_t;
      const int least = wave_min(key);
      if (least < qj) {
        const int s = __builtin_ctzll(__ballot(key == least));
        if (least >= 0) flush(s, __builtin_amdgcn_readlane(slot_id, s));
        if (lane == i) code = s;
        if (lane == s) {
          slot_id = uniform_int(mb.ctx[i]);
          slot_t = qj;
        }
      }
    }
  }
  if (lane < n) mb.slot[lane] = code;
  __syncthreads();
}

// Waves per SIMD the register allocation must allow, where the default
// allocation lands just above a residency step. With several output blocks
// at C <= 2 (178 registers, 2 waves) a bound of 3 spills three registers;
// with one block at C = 4 (175, 2 waves) a bound of 3 spills two, and at
// C = 10 (256 + 20, 1 wave) a bound of 2 spills 26. Each measured faster
// (D = 100, K = 15: +9%; D = 200, K = 5: +5%; D = 600, K = 5: +19%). The
// bounds apply to the kernels of up to 10 input words (window <= 5);
// elsewhere, and at C = 5 (3 waves: 29 spills, no LDS left for pending
// rows, -8%), the next step up costs more than it gains.
template <int C, int NMAX, bool kMulti>
constexpr int epoch_waves_per_eu() {
  if (NMAX > 10) return 1;
  if (kMulti) return C <= 2 ? 3 : 1;
  return C == 4 ? 3 : (C >= 10 ? 2 : 1);
}

template <int C, int NMAX, bool kMulti, bool kExport>
__global__ __launch_bounds__(kWave) __attribute__((
    amdgpu_waves_per_eu(epoch_waves_per_eu<C, NMAX, kMulti>()))) void k_epoch(EpochArgs a) {
  __shared__ SentenceLds sl;
  __shared__ TargetBatch tb;
  __shared__ MinibatchLds mb;
  extern __shared__ int32_t negs_lds[];  // [TB][K], then the pending slots
  const int lane = threadIdx.x;
  const int K = a.K;
  const bool want_loss = a.loss != nullptr;
  const int TB = kExport ? kWave : a.target_batch;  // targets formed at once
  float* const slot_rows = reinterpret_cast<float*>(negs_lds + TB * (K > 0 ? K : 1));
  const int nslots = kExport ? 0 : a.pend_slots;
  int slot_id = -1, slot_t = 0;
  const RowTiers<C, false> io{a.part, a.split_rows, a.hot_rows, a.ld, a.D, lane};
  // Adds the pending updates of slot s to the M_in row of word id.
  auto flush = [&](int s, int id) {
    const float* p = slot_rows + s * (kWave * C) + lane;
    float d[C];
#pragma unroll
    for (int c = 0; c < C; ++c) d[c] = p[kWave * c];
    io.add(0, a.M_in, id, d);
  };

  int64_t n_mb = 0, sum_n = 0, raw = 0, rejected = 0, rows = 0;
  double lsum = 0.0, lcnt = 0.0;
  int bucket = -1;

  for (int64_t s = blockIdx.x; s < a.n_sent; s += gridDim.x) {
    const int64_t sb = a.pos_begin + s * a.L;
    const int64_t se = min(sb + (int64_t)a.L, a.pos_end);
    const int len = (int)(se - sb);
    raw += len;
    const int n_ret = keep_and_compact<kExport>(a, sb, len, lane, sl, rejected);

    for (int q0 = 0; q0 < n_ret; q0 += TB) {
      form_targets<kExport>(a, sb, q0, n_ret, lane, sl, tb, negs_lds, TB);
      const int cnt = min(TB, n_ret - q0);
      for (int j = 0; j < cnt; ++j) {
        const int n = uniform_int(tb.n[j]);
        if (n == 0) continue;
        if (uniform_int(tb.bad[j]) != 0) {
          ++rejected;
          continue;
        }
        ++n_mb;
        sum_n += n;
        if constexpr (!kExport) {
          const int qj = q0 + j;
          const int lo = uniform_int(tb.lo[j]);
          int ctx_id = 0;
          if (lane < n) {
            int jj = lo + lane;
            if (jj >= qj) ++jj;
            ctx_id = sl.ret_id[jj];
          }
          const int n_in = stage_inputs(lane, ctx_id, lane < n, mb);
          const int neg = lane < K ? negs_lds[j * K + lane] : 0;
          const int n_out = stage_outputs(lane, sl.ret_id[qj], neg, K, mb);
          rows += n_in + n_out;
          if (nslots > 0)
            assign_slots<NMAX>(mb, n_in, qj, 2 * a.w, nslots, a.pend_from, lane,
                               slot_id, slot_t, flush);
          else if (lane < n_in)
            mb.slot[lane] = -1;
          const PendingRows pend{slot_rows, mb.slot};
          float loss_part = 0.f;
          run_minibatch<C, NMAX, kMulti, true, false>(
              a.M_in, a.M_out, a.M_in, a.M_out, a.ld, a.D, lane, n_in, n_out,
              uniform_float(tb.alpha[j]), a.hot_rows, mb, want_loss,
              loss_part, a.part, a.split_rows, TargetError(), pend);
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
    if constexpr (!kExport) {
      for (uint64_t held = __ballot(lane < nslots && slot_id >= 0); held != 0ull;
           held &= held - 1ull) {
        const int s = __builtin_ctzll(held);
        flush(s, __builtin_amdgcn_readlane(slot_id, s));
      }
      slot_id = -1;
    }
  }
  if (want_loss && bucket >= 0) flush_loss(a.loss, bucket, lsum, lcnt, lane);
  flush_stats(a, lane, n_mb, sum_n, raw, rejected, rows);
}

// Partial rows of the split rows: cleared before an epoch, summed (in the
// order g = 0, 1, ...) and added into the matrices with one rounding, then
// cleared, after it; a row with nothing pending keeps its bits. One thread
// per (matrix, row, column).
__global__ __launch_bounds__(256) void k_part_clear(EpochArgs a) {
  const int64_t n = (int64_t)2 * a.split_rows * kSplitParts * a.ld;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    a.part[i] = 0.f;
}

__global__ __launch_bounds__(256) void k_part_fold(EpochArgs a) {
  const int64_t n = (int64_t)2 * a.split_rows * a.D;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int col = (int)(i % a.D);
    const int64_t mr = i / a.D;  // m * split_rows + row
    const int m = (int)(mr / a.split_rows);
    const int64_t row = mr % a.split_rows;
    float* pb = a.part + mr * kSplitParts * a.ld + col;
    float* dst = (m == 0 ? a.M_in : a.M_out) + row * a.ld + col;
    float sum = 0.f;
    for (int g = 0; g < kSplitParts; ++g) {
      sum += pb[g * a.ld];
      pb[g * a.ld] = 0.f;
    }
    if (sum != 0.f) *dst += sum;
  }
}

// The same epoch with the K negatives shared by groups of G consecutive
// targets (group_core.h): per group, the members' input occurrences and the
// output candidates (member targets, then the group's negatives) are staged
// deduplicated with their group tables, then one snapshot step runs over the
// group (group_core.h) with up to OMAX output columns. Groups start at
// retained indices that are multiples of G (G divides the 64-target
// batches).
template <int C, int OMAX>
__global__ __launch_bounds__(kWave) void k_epoch_grouped(EpochArgs a) {
  __shared__ SentenceLds sl;
  __shared__ TargetBatch tb;
  __shared__ MinibatchLds mb;
  __shared__ GroupLds gl;
  extern __shared__ int32_t negs_lds[];  // [kWave][K]
  const int lane = threadIdx.x;
  const int K = a.K;
  const int G = a.group;
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
      for (int j0 = 0; j0 < cnt; j0 += G) {
        // Members: lane g < G holds the input count of target j0 + g.
        const int n_g = (lane < G && j0 + lane < cnt) ? tb.n[j0 + lane] : 0;
        const uint64_t members = __ballot(n_g > 0);
        if (members == 0ull) continue;
        if (uniform_int(tb.bad[j0]) != 0) {
          rejected += __popcll(members);
          continue;
        }
        // Input occurrences, member by member, one per lane.
        int off = 0, my_g = -1, my_i = 0;
#pragma unroll
        for (int g = 0; g < kMaxGroup; ++g) {
          if (g < G) {
            const int ng = __builtin_amdgcn_readlane(n_g, g);
            if (lane >= off && lane < off + ng) {
              my_g = g;
              my_i = lane - off;
            }
            off += ng;
          }
        }
        const int total = off;
        if (my_g >= 0) {
          const int q = q0 + j0 + my_g;
          int jj = tb.lo[j0 + my_g] + my_i;
          if (jj >= q) ++jj;
          gl.occ_id[lane] = sl.ret_id[jj];
          gl.occ_g[lane] = my_g;
        }
        if (lane < G)
          gl.alpha[lane] = n_g > 0 ? tb.alpha[j0 + lane] : 0.f;
        // Output candidates: member targets, then the group's negatives
        // (drawn at its first retained position).
        int cid = -1;
        if (lane < G) {
          if (n_g > 0) cid = sl.ret_id[q0 + j0 + lane];
        } else if (lane < G + K) {
          cid = negs_lds[j0 * K + (lane - G)];
        }
        gl.cand_id[lane] = cid;
        __syncthreads();

        // Distinct input rows and their multiplicity per member.
        const int my_id = my_g >= 0 ? gl.occ_id[lane] : -1;
        bool first = my_g >= 0;
        float mult[kMaxGroup];
#pragma unroll
        for (int g = 0; g < kMaxGroup; ++g) mult[g] = 0.f;
        if (my_g >= 0) {
          for (int l2 = 0; l2 < total; ++l2) {
            if (gl.occ_id[l2] != my_id) continue;
            if (l2 < lane) first = false;
            const int g2 = gl.occ_g[l2];
#pragma unroll
            for (int g = 0; g < kMaxGroup; ++g) mult[g] += (g2 == g) ? 1.f : 0.f;
          }
        }
        const uint64_t fin = __ballot(first);
        if (first) {
          const int dst = __popcll(fin & lanes_below(lane));
          mb.ctx[dst] = my_id;
#pragma unroll
          for (int g = 0; g < kMaxGroup; ++g) gl.m[dst][g] = mult[g];
        }
        const int n_in = __popcll(fin);

        // Distinct output columns: member-target bits and negative weight.
        bool cfirst = cid >= 0;
        uint32_t bits = 0u;
        float nw = 0.f;
        if (cid >= 0) {
          for (int c2 = 0; c2 < G + K; ++c2) {
            if (gl.cand_id[c2] != cid) continue;
            if (c2 < lane) cfirst = false;
            if (c2 < G) bits |= 1u << c2;
            else nw += 1.f;
          }
        }
        const uint64_t fout = __ballot(cfirst);
        if (cfirst) {
          const int dst = __popcll(fout & lanes_below(lane));
          mb.out[dst] = cid;
          gl.tbits[dst] = bits;
          gl.negw[dst] = nw;
        }
        const int n_out = __popcll(fout);
        __syncthreads();

        n_mb += __popcll(members);
        sum_n += total;
        rows += n_in + n_out;
        float loss_part = 0.f;
        run_group<C, OMAX>(a, lane, n_in, n_out, mb, gl, G, want_loss, loss_part);
        if (want_loss) {
          const int qf = q0 + j0 + (int)__builtin_ctzll(members);
          const int64_t p = sb + sl.ret_off[qf];
          const int b = (int)(p * (int64_t)a.n_buckets / a.T);
          if (b != bucket) {
            if (bucket >= 0) flush_loss(a.loss, bucket, lsum, lcnt, lane);
            bucket = b;
          }
          lsum += (double)loss_part;
          if (lane == 0) lcnt += (double)total;
        }
        __syncthreads();
      }
      __syncthreads();
    }
  }
  if (want_loss && bucket >= 0) flush_loss(a.loss, bucket, lsum, lcnt, lane);
  flush_stats(a, lane, n_mb, sum_n, raw, rejected, rows);
}

// ------------------------------------------------------------ launchers --

static int part_grid(int64_t n) {
  const int64_t b = (n + 255) / 256;
  return (int)(b < 4096 ? (b > 0 ? b : 1) : 4096);
}

hipError_t launch_part_clear(const EpochArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_part_clear,
                     dim3(part_grid((int64_t)2 * a.split_rows * kSplitParts * a.ld)),
                     dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_part_fold(const EpochArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_part_fold, dim3(part_grid((int64_t)2 * a.split_rows * a.D)),
                     dim3(256), 0, s, a);
  return hipGetLastError();
}

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

// gfx950 gives each CU 160 KB of LDS and allocates it to a workgroup in
// granules of 1280 bytes. The runtime's occupancy query admits requests that
// the granules do not: at D = 100, K = 5 it allowed 12 workgroups per CU
// with 12,808 bytes each, 12 x 10 granules would need 168,960 bytes, and a
// twelfth of the persistent grid then waited for a free CU (-34%
// throughput). Both limits apply.
constexpr size_t kLdsPerCu = 160 * 1024;
constexpr size_t kLdsGranule = 1280;

int resident_blocks_per_cu(const void* kernel, size_t dyn_lds) {
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, kernel, kWave,
                                                   dyn_lds) != hipSuccess)
    return 0;
  hipFuncAttributes attr{};
  if (hipFuncGetAttributes(&attr, kernel) != hipSuccess) return 0;
  const size_t per = (attr.sharedSizeBytes + dyn_lds + kLdsGranule - 1) /
                     kLdsGranule * kLdsGranule;
  const int by_lds = (int)(kLdsPerCu / per);
  return blocks < by_lds ? blocks : by_lds;
}

static size_t negatives_lds(int K, int batch = kWave) {
  return sizeof(int32_t) * (size_t)batch * (size_t)(K > 0 ? K : 1);
}

static size_t epoch_dyn_lds(const EpochArgs& a) {
  return negatives_lds(a.K);
}

static size_t slot_bytes(int C) { return sizeof(float) * (size_t)kWave * C; }

constexpr int kMaxPendingSlots = 16;

// Shape of the training launch for (C, nmax, K) on the current device:
// targets formed at once, pending slots and resident workgroups per CU.
// Computed from occupancy queries once per device and shape.
struct TrainShape {
  int target_batch, pending_slots, blocks_per_cu;
};

static TrainShape compute_train_shape(int C, int nmax, int K) {
  TrainShape t{kWave, 0, 0};
  EpochKernel k = train_kernel_for(C, nmax, K);
  if (k == nullptr) return t;
  const void* f = reinterpret_cast<const void*>(k);
  const int best = resident_blocks_per_cu(f, negatives_lds(K, 8));
  while (t.target_batch > 8 &&
         resident_blocks_per_cu(f, negatives_lds(K, t.target_batch)) < best)
    t.target_batch /= 2;
  const size_t negs = negatives_lds(K, t.target_batch);
  t.blocks_per_cu = resident_blocks_per_cu(f, negs);
  if (t.blocks_per_cu <= 0) return t;
  for (int n = kMaxPendingSlots; n >= 2; --n)
    if (resident_blocks_per_cu(f, negs + n * slot_bytes(C)) >= t.blocks_per_cu) {
      t.pending_slots = n;
      break;
    }
  return t;
}

static TrainShape train_shape(int C, int nmax, int K) {
  static std::mutex mu;
  static std::map<std::tuple<int, int, int, int>, TrainShape> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return compute_train_shape(C, nmax, K);
  const auto key = std::make_tuple(dev, C, nmax, K);
  std::lock_guard<std::mutex> lock(mu);
  auto it = cache.find(key);
  if (it != cache.end()) return it->second;
  const TrainShape t = compute_train_shape(C, nmax, K);
  if (t.blocks_per_cu > 0) cache[key] = t;  // failed queries are retried
  return t;
}

int train_target_batch(int C, int nmax, int K) { return train_shape(C, nmax, K).target_batch; }

int train_pending_slots(int C, int nmax, int K) { return train_shape(C, nmax, K).pending_slots; }

int train_blocks_per_cu(int C, int nmax, int K) { return train_shape(C, nmax, K).blocks_per_cu; }

hipError_t launch_train(int C, int nmax, const EpochArgs& a, int grid,
                        hipStream_t s) {
  EpochKernel k = train_kernel_for(C, nmax, a.K);
  if (k == nullptr) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k, dim3(grid), dim3(kWave),
                     negatives_lds(a.K, a.target_batch) + a.pend_slots * slot_bytes(C),
                     s, a);
  return hipGetLastError();
}

#define W2V_GROUP_SHAPES(X) \
  X(1, 10) X(2, 10) X(3, 10) X(4, 10) X(5, 10) X(6, 10) X(8, 10) X(10, 10) \
  X(1, 16) X(2, 16) X(3, 16) X(4, 16) X(5, 16) X(6, 16) X(1, 32) X(2, 32)

static EpochKernel grouped_kernel_for(int C, int omax) {
#define W2V_PICK(c, n) \
  if (C == c && omax == n) return k_epoch_grouped<c, n>;
  W2V_GROUP_SHAPES(W2V_PICK)
#undef W2V_PICK
  return nullptr;
}

int group_outputs_cap_for(int n) {
  if (n <= 10) return 10;
  if (n <= 16) return 16;
  if (n <= 32) return 32;
  return 0;
}

bool grouped_shape_supported(int C, int omax) {
  return grouped_kernel_for(C, omax) != nullptr;
}

int grouped_blocks_per_cu(int C, int omax, int K) {
  EpochKernel k = grouped_kernel_for(C, omax);
  if (k == nullptr) return 0;
  return resident_blocks_per_cu(reinterpret_cast<const void*>(k), negatives_lds(K));
}

hipError_t launch_grouped(int C, int omax, const EpochArgs& a, int grid,
                          hipStream_t s) {
  EpochKernel k = grouped_kernel_for(C, omax);
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
