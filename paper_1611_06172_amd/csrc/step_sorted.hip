// Sorted snapshot batch on gfx950: the step of the atomic snapshot batch
// (step_kernels.hip) with every row's updates summed in one fixed order, so
// that a batch gives the same bits on every run and no atomics are needed.
//
//   1. k_stage: one wavefront per minibatch computes its updates from the
//      unchanged matrices (sgns_core.h) and writes them to staging rows
//      (StagedRows) instead of applying them. Each staging row gets a sort
//      key naming the matrix row it updates: id for M_in, V + id for M_out,
//      2V for an unused staging row;
//   2. one stable radix sort of (key, staging index) pairs (radix_sort.hip),
//      so each matrix row's updates form one run, in minibatch order;
//   3. k_reduce: one wavefront per chunk of 64 sorted entries sums each run
//      it holds in fp64, in sorted order, loading kBatch staging rows (and
//      the matrix rows of the runs that open among them) at once. A run
//      inside the chunk is applied (M = fp32(M + sum) where the sum is not
//      0); the part of a run that crosses the chunk's first or last border
//      goes to the chunk's head or tail piece;
//   4. k_reduce_spans: a run's head pieces within one span of kSpan chunks
//      are added, in chunk order, into the first of them;
//   5. k_reduce_cross: the chunk in which a crossing run starts finds the
//      run's last chunk (galloping search over chunk borders), adds its
//      tail piece and the run's summed piece of every span it goes through,
//      in span order, and applies the total.
// Traffic per batch: the gathered rows, one staging row written and read
// per update, the keys, and one read and write per touched row.
#include <hip/hip_runtime.h>

#include "kernel_args.h"
#include "sgns_core.h"

namespace w2v {

constexpr int kChunk = 64;   // sorted entries per wavefront (one per lane)
constexpr int kBatch = 8;    // rows loaded before they are added

template <int C, int NMAX, bool kMulti>
__global__ __launch_bounds__(kWave) void k_stage(SortedStepArgs a) {
  __shared__ MinibatchLds mb;
  const int lane = threadIdx.x;
  const int n_slots_out = a.K + 1;
  int64_t applied = 0, sum_n = 0, rejected = 0, rows = 0;
  for (int64_t b = blockIdx.x; b < a.B; b += gridDim.x) {
    const int t = a.targets[b];
    int bad = (t < 0 || t >= a.V);
    int c = -1;
    if (lane < a.N) c = a.contexts[b * a.N + lane];
    bad |= (c < -1 || c >= a.V);
    const bool present = c >= 0;
    const int n = __popcll(__ballot(present));
    const int n_in = stage_inputs(lane, c, present, mb);
    int neg = 0;
    if (lane < a.K) {
      neg = a.negatives[b * a.K + lane];
      bad |= (neg < 0 || neg >= a.V);
    }
    const bool any_bad = __ballot(bad != 0) != 0ull;
    const int n_out = stage_outputs(lane, t, neg, a.K, mb);
    const bool use = !any_bad && n > 0;
    // Keys of this minibatch's staging rows (2V where nothing is staged).
    const int64_t in0 = b * a.N, out0 = b * n_slots_out;
    const uint32_t unused = 2u * (uint32_t)a.V;
    if (lane < a.N) {
      a.key_in[in0 + lane] = (use && lane < n_in) ? (uint32_t)mb.ctx[lane] : unused;
      a.val_in[in0 + lane] = (int32_t)(in0 + lane);
    }
    for (int k = lane; k < n_slots_out; k += kWave) {
      a.key_out[out0 + k] =
          (use && k < n_out) ? (uint32_t)a.V + (uint32_t)mb.out[k] : unused;
      a.val_out[out0 + k] = (int32_t)(a.out_base + out0 + k);
    }
    if (any_bad) {
      ++rejected;
    } else if (n > 0) {
      ++applied;
      sum_n += n;
      rows += n_in + n_out;
      const float alpha = a.alpha != nullptr ? a.alpha[b] : a.alpha_scalar;
      float unused = 0.f;
      const StagedRows stage{a.stage_in + in0 * a.ld, a.stage_out + out0 * a.ld,
                             a.ld, a.D};
      run_minibatch<C, NMAX, kMulti, false, false, TargetError, StagedRows>(
          a.M_in, a.M_out, a.M_in, a.M_out, a.ld, a.D, lane, n_in, n_out, alpha,
          0, mb, false, unused, nullptr, 0, TargetError(), stage);
    }
    __syncthreads();
  }
  if (lane == 0) report_bad_ids(a.status, rejected);
  if (a.stats != nullptr && lane == 0) {
    atomicAdd((unsigned long long*)&a.stats[0], (unsigned long long)applied);
    atomicAdd((unsigned long long*)&a.stats[1], (unsigned long long)sum_n);
    atomicAdd((unsigned long long*)&a.stats[3], (unsigned long long)rejected);
    atomicAdd((unsigned long long*)&a.stats[4], (unsigned long long)rows);
  }
}

// The sorted updates of both matrices: n entries (key, staging index),
// staging rows of stride ld, pieces[(2 chunk + h) ld] (h = 0 head, 1 tail).
struct ReduceArgs {
  const uint32_t* key;
  const int32_t* val;
  int64_t n;
  const float* stage;
  float* M_in;
  float* M_out;
  double* pieces;          // [2 n_chunks][pstride], pstride >= 64 C
  int32_t V, D;
  int64_t ld, pstride;
};

// Matrix row a sort key names (keys < 2V).
__device__ __forceinline__ float* key_row(const ReduceArgs& r, uint32_t key) {
  return key < (uint32_t)r.V ? r.M_in + (int64_t)key * r.ld
                             : r.M_out + (int64_t)(key - (uint32_t)r.V) * r.ld;
}

template <int C>
__device__ __forceinline__ void apply_sum(const ReduceArgs& r, uint32_t key,
                                          int lane, const double (&sum)[C]) {
  float* row = key_row(r, key);
  float m[C];
  load_row<C, false>(row, 0, r.ld, r.D, lane, m);
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int col = lane + kWave * c;
    if (col < r.D && sum[c] != 0.0) row[col] = (float)((double)m[c] + sum[c]);
  }
}

// Piece rows hold all 64 C columns (zero past D), so they are written and
// read without per-column tests.
template <int C>
__device__ __forceinline__ void put_piece(const ReduceArgs& r, int64_t chunk,
                                          int h, int lane,
                                          const double (&sum)[C]) {
  double* p = r.pieces + (2 * chunk + h) * r.pstride + lane;
#pragma unroll
  for (int c = 0; c < C; ++c) p[kWave * c] = sum[c];
}

// Lane's columns of the n_bytes-long row at p (range-checked loads: 0 past
// the end, all 0 for n_bytes = 0), issued without a branch so that a batch
// of them stays in flight together.
template <int C>
__device__ __forceinline__ void load_masked(const float* p, int n_bytes, int lane,
                                            float (&x)[C]) {
  const __amdgpu_buffer_rsrc_t rs = row_rsrc(p, n_bytes);
#pragma unroll
  for (int c = 0; c < C; ++c)
    x[c] = __uint_as_float(
        __builtin_amdgcn_raw_buffer_load_b32(rs, (lane + kWave * c) * 4, 0, 0));
}

template <int C>
__global__ __launch_bounds__(kWave) void k_reduce(ReduceArgs r) {
  const int lane = threadIdx.x;
  const int64_t n_chunks = (r.n + kChunk - 1) / kChunk;
  static_assert(kChunk == kWave, "one sorted entry per lane");
  for (int64_t ch = blockIdx.x; ch < n_chunks; ch += gridDim.x) {
    const int64_t lo = ch * kChunk;
    const int cnt = (int)(lo + kChunk < r.n ? kChunk : r.n - lo);
    // The chunk's keys and staging indices, one per lane.
    const uint32_t kl = lane < cnt ? r.key[lo + lane] : 0xffffffffu;
    const int32_t vl = lane < cnt ? r.val[lo + lane] : 0;
    const uint32_t prev = lo > 0 ? r.key[lo - 1] : 0xffffffffu;
    const uint32_t next = lo + cnt < r.n ? r.key[lo + cnt] : 0xffffffffu;
    uint32_t cur = 0xffffffffu;  // key of the open run (none yet)
    int start = 0, end = cnt;
    double sum[C];
    float mrow[C];               // matrix row of the open run, as read
#pragma unroll
    for (int c = 0; c < C; ++c) {
      sum[c] = 0.0;
      mrow[c] = 0.f;
    }
    // Closes the run [s, e) of key k: applied, or left as the chunk's head
    // piece (it began in an earlier chunk) or tail piece (it goes on).
    auto close = [&](uint32_t k, int s, int e) {
      if (s == 0 && prev == k) {
        put_piece<C>(r, ch, 0, lane, sum);
      } else if (e == cnt && next == k) {
        put_piece<C>(r, ch, 1, lane, sum);
      } else {
        float* row = key_row(r, k);
#pragma unroll
        for (int c = 0; c < C; ++c) {
          const int col = lane + kWave * c;
          if (col < r.D && sum[c] != 0.0) row[col] = (float)((double)mrow[c] + sum[c]);
        }
      }
    };
    bool done = false;
    for (int j0 = 0; j0 < cnt && !done; j0 += kBatch) {
      // Issue a batch of staging-row loads, and the matrix row of every run
      // that opens in the batch, then add them in order. A run's matrix row
      // is written by no one else before this wavefront applies it.
      float x[kBatch][C], m[kBatch][C];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int j = j0 + u;
        const uint32_t k = (uint32_t)__builtin_amdgcn_readlane((int)kl, j);
        const uint32_t kp = j == 0 ? prev : (uint32_t)__builtin_amdgcn_readlane((int)kl, j - 1);
        const bool valid = j < cnt && k < 2u * (uint32_t)r.V;
        const int32_t v = __builtin_amdgcn_readlane(vl, j);
        load_masked<C>(r.stage + (int64_t)(valid ? v : 0) * r.ld, valid ? r.D * 4 : 0,
                       lane, x[u]);
        const bool opens = valid && k != kp;
        load_masked<C>(key_row(r, opens ? k : 0u), opens ? r.D * 4 : 0, lane, m[u]);
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int j = j0 + u;
        const uint32_t k = (uint32_t)__builtin_amdgcn_readlane((int)kl, j);
        if (done || j >= cnt || k >= 2u * (uint32_t)r.V) {
          if (!done) end = j;
          done = true;
        } else {
          if (k != cur) {
            if (cur != 0xffffffffu) close(cur, start, j);
            cur = k;
            start = j;
#pragma unroll
            for (int c = 0; c < C; ++c) {
              sum[c] = 0.0;
              mrow[c] = m[u][c];
            }
          }
#pragma unroll
          for (int c = 0; c < C; ++c) sum[c] += (double)x[u][c];
        }
      }
    }
    if (cur != 0xffffffffu) close(cur, start, end);
  }
}

// Chunks per span: the head pieces of one run inside one span of kSpan
// chunks are first added into the span's first such piece, so that a run
// over many chunks costs its start chunk one read per span.
constexpr int kSpan = 32;

// Key of the first entry of chunk c, and whether its run began earlier.
__device__ __forceinline__ bool has_head(const ReduceArgs& r, int64_t c,
                                         uint32_t& key) {
  const int64_t lo = c * kChunk;
  if (lo <= 0 || lo >= r.n) return false;
  key = r.key[lo];
  return key < 2u * (uint32_t)r.V && r.key[lo - 1] == key;
}

// Adds `count` piece rows at pieces[2 (c0 + i)] (i < count), a batch at a
// time, in order.
template <int C>
__device__ __forceinline__ void add_heads(const ReduceArgs& r, int64_t c0,
                                          int64_t count, int lane,
                                          double (&sum)[C]) {
  for (int64_t i0 = 0; i0 < count; i0 += kBatch) {
    double x[kBatch][C];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      // past the end: re-read the last piece, not added below
      const int64_t cu = c0 + (i0 + u < count ? i0 + u : count - 1);
      const double* head = r.pieces + 2 * cu * r.pstride + lane;
#pragma unroll
      for (int c = 0; c < C; ++c) x[u][c] = head[kWave * c];
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
      if (i0 + u < count)
#pragma unroll
        for (int c = 0; c < C; ++c) sum[c] += x[u][c];
  }
}

// For every (run, span) with head pieces, the wavefront of the first such
// chunk adds the run's head pieces in the span, in chunk order, into that
// chunk's head piece.
template <int C>
__global__ __launch_bounds__(kWave) void k_reduce_spans(ReduceArgs r) {
  const int lane = threadIdx.x;
  const int64_t n_chunks = (r.n + kChunk - 1) / kChunk;
  for (int64_t ch = blockIdx.x; ch < n_chunks; ch += gridDim.x) {
    uint32_t key;
    if (!has_head(r, ch, key)) continue;
    uint32_t kp;
    if (ch % kSpan != 0 && has_head(r, ch - 1, kp) && kp == key) continue;
    // The run's head pieces in this span: chunks ch, ch+1, ... (lane j
    // tests chunk ch + 1 + j; the run's chunks are consecutive).
    const int64_t span_end = (ch / kSpan + 1) * kSpan;
    const int64_t cj = ch + 1 + lane;
    uint32_t kj = 0u;
    const bool same = cj < span_end && has_head(r, cj, kj) && kj == key;
    const int64_t end = ch + 1 + __builtin_ctzll(~__ballot(same));
    if (end == ch + 1) continue;  // a single head piece is its own sum
    double sum[C];
#pragma unroll
    for (int c = 0; c < C; ++c) sum[c] = 0.0;
    add_heads<C>(r, ch, end - ch, lane, sum);
    put_piece<C>(r, ch, 0, lane, sum);
  }
}

template <int C>
__global__ __launch_bounds__(kWave) void k_reduce_cross(ReduceArgs r) {
  const int lane = threadIdx.x;
  const int64_t n_chunks = (r.n + kChunk - 1) / kChunk;
  for (int64_t ch = blockIdx.x; ch < n_chunks; ch += gridDim.x) {
    const int64_t lo = ch * kChunk;
    const int64_t hi = lo + kChunk;
    if (hi >= r.n) continue;
    const uint32_t key = r.key[hi - 1];
    if (key >= 2u * (uint32_t)r.V || r.key[hi] != key) continue;
    // The run continues into the next chunk; it starts in this one unless
    // the whole chunk belongs to a run that began earlier.
    if (lo > 0 && r.key[lo] == key && r.key[lo - 1] == key) continue;
    // Last chunk of the run: the chunk ch + d is inside the run when the
    // entry opening it still has the key; gallop over d = 1, 2, 4, ... and
    // bisect, so a run over P chunks costs about 2 log2 P key reads.
    auto inside = [&](int64_t d) {
      const int64_t e = (ch + d) * kChunk;
      return e < r.n && r.key[e] == key;
    };
    int64_t good = 1, step = 1;      // chunk ch + 1 holds part of the run
    while (inside(good + step)) {
      good += step;
      step *= 2;
    }
    int64_t bad = good + step;       // first d known outside
    while (bad - good > 1) {
      const int64_t mid = good + (bad - good) / 2;
      if (inside(mid)) good = mid; else bad = mid;
    }
    const int64_t last_chunk = ch + good;
    double sum[C];
    const double* tail = r.pieces + (2 * ch + 1) * r.pstride + lane;
#pragma unroll
    for (int c = 0; c < C; ++c) sum[c] = tail[kWave * c];
    // One summed piece per span the run goes through (k_reduce_spans), in
    // span order: the first at ch + 1, the others at span starts.
    const int64_t first_span = (ch + 1) / kSpan, last_span = last_chunk / kSpan;
    for (int64_t sp0 = first_span; sp0 <= last_span; sp0 += kBatch) {
      double x[kBatch][C];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int64_t sp = sp0 + u <= last_span ? sp0 + u : last_span;
        const int64_t c1 = sp == first_span ? ch + 1 : sp * kSpan;
        const double* head = r.pieces + 2 * c1 * r.pstride + lane;
#pragma unroll
        for (int c = 0; c < C; ++c) x[u][c] = head[kWave * c];
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u)
        if (sp0 + u <= last_span)
#pragma unroll
          for (int c = 0; c < C; ++c) sum[c] += x[u][c];
    }
    apply_sum<C>(r, key, lane, sum);
  }
}

#define W2V_SORTED_SHAPES(X) \
  X(1, 10) X(2, 10) X(3, 10) X(4, 10) X(5, 10) X(6, 10) X(8, 10) X(10, 10) \
  X(1, 16) X(2, 16) X(3, 16) X(4, 16) X(5, 16) X(1, 32) X(2, 32)

using StageKernel = void (*)(SortedStepArgs);
using ReduceKernel = void (*)(ReduceArgs);

static StageKernel stage_kernel_for(int C, int nmax, int K) {
  const bool multi = K + 1 > kWave / nmax;
#define W2V_PICK(c, n) \
  if (C == c && nmax == n) return multi ? k_stage<c, n, true> : k_stage<c, n, false>;
  W2V_SORTED_SHAPES(W2V_PICK)
#undef W2V_PICK
  return nullptr;
}

static bool reduce_kernels_for(int C, ReduceKernel& red, ReduceKernel& spans,
                               ReduceKernel& cross) {
  switch (C) {
#define W2V_CASE(c) \
  case c:           \
    red = k_reduce<c>; spans = k_reduce_spans<c>; cross = k_reduce_cross<c>; return true;
    W2V_CASE(1) W2V_CASE(2) W2V_CASE(3) W2V_CASE(4) W2V_CASE(5) W2V_CASE(6)
    W2V_CASE(8) W2V_CASE(10)
#undef W2V_CASE
    default:
      return false;
  }
}

static size_t align256(size_t x) { return (x + 255) / 256 * 256; }

static int key_bits(int32_t V) {
  return 32 - __builtin_clz(2u * (unsigned)V);  // keys are 0..2V
}

// Temporary bytes of the sort of n pairs.
static bool sort_temp_bytes(int64_t n, int32_t V, size_t& bytes) {
  (void)V;
  bytes = radix_sort_temp_bytes(n, sizeof(uint32_t));
  return true;
}

// Doubles per piece row: at least 64 C for the C a row stride of ld can
// need (D <= ld; C = ceil(D/64) rounded up to a compiled size, at most one
// more).
static int64_t piece_stride(int32_t ld) { return (int64_t)kWave * ((ld + kWave - 1) / kWave + 1); }

// Workspace: staging rows (inputs, then outputs), keys, sorted keys,
// values, sorted values, pieces, sort temporaries.
struct SortedLayout {
  int64_t n_in, n;
  size_t stage, ints, pieces, temp, total;
  bool ok;
};

static SortedLayout sorted_layout(int32_t B, int32_t N, int32_t K, int32_t V,
                                  int32_t ld) {
  SortedLayout L{};
  L.n_in = (int64_t)B * N;
  L.n = L.n_in + (int64_t)B * (K + 1);
  L.stage = align256(sizeof(float) * (size_t)L.n * ld);
  L.ints = align256(sizeof(uint32_t) * (size_t)L.n);
  L.pieces = align256(sizeof(double) * 2 * (size_t)((L.n + kChunk - 1) / kChunk) *
                     (size_t)piece_stride(ld));
  size_t t = 0;
  L.ok = sort_temp_bytes(L.n, V, t);
  L.temp = align256(t);
  L.total = L.stage + 4 * L.ints + L.pieces + L.temp;
  if (L.total == 0) L.total = 256;
  return L;
}

size_t sorted_step_workspace_bytes(int32_t B, int32_t N, int32_t K, int32_t V,
                                   int32_t ld) {
  const SortedLayout L = sorted_layout(B, N, K, V, ld);
  return L.ok ? L.total : 0;
}

bool sorted_step_supported(int C, int nmax) {
  ReduceKernel r, sp, x;
  return stage_kernel_for(C, nmax, 0) != nullptr && reduce_kernels_for(C, r, sp, x);
}

hipError_t launch_step_sorted(int C, int nmax, SortedStepArgs a, void* workspace,
                              hipStream_t s) {
  StageKernel k = stage_kernel_for(C, nmax, a.K);
  ReduceKernel red, spans, cross;
  if (k == nullptr || !reduce_kernels_for(C, red, spans, cross)) return hipErrorInvalidValue;
  const SortedLayout L = sorted_layout(a.B, a.N, a.K, a.V, (int32_t)a.ld);
  char* w = (char*)workspace;
  float* stage = (float*)w;
  uint32_t* keys = (uint32_t*)(w + L.stage);
  uint32_t* keys_sorted = (uint32_t*)(w + L.stage + L.ints);
  int32_t* vals = (int32_t*)(w + L.stage + 2 * L.ints);
  int32_t* vals_sorted = (int32_t*)(w + L.stage + 3 * L.ints);
  double* pieces = (double*)(w + L.stage + 4 * L.ints);
  void* temp = (void*)(w + L.stage + 4 * L.ints + L.pieces);
  a.stage_in = stage;
  a.stage_out = stage + L.n_in * a.ld;
  a.key_in = keys;
  a.val_in = vals;
  a.key_out = keys + L.n_in;
  a.val_out = vals + L.n_in;
  a.out_base = L.n_in;
  const int grid = a.B < (1 << 20) ? a.B : (1 << 20);
  hipLaunchKernelGGL(k, dim3(grid), dim3(kWave), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = radix_sort_pairs((const uint32_t*)keys, (const int32_t*)vals, keys_sorted,
                       vals_sorted, L.n, key_bits(a.V), temp, s);
  if (e != hipSuccess) return e;
  ReduceArgs r{keys_sorted, vals_sorted, L.n, stage, a.M_in, a.M_out, pieces,
               a.V, a.D, a.ld, piece_stride((int32_t)a.ld)};
  if (r.pstride < (int64_t)kWave * C) return hipErrorInvalidValue;
  const int64_t n_chunks = (L.n + kChunk - 1) / kChunk;
  const int rgrid = (int)(n_chunks < 65536 ? n_chunks : 65536);
  hipLaunchKernelGGL(red, dim3(rgrid), dim3(kWave), 0, s, r);
  hipLaunchKernelGGL(spans, dim3(rgrid), dim3(kWave), 0, s, r);
  hipLaunchKernelGGL(cross, dim3(rgrid), dim3(kWave), 0, s, r);
  return hipGetLastError();
}

}  // namespace w2v
