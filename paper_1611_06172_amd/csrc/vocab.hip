// Vocabulary of a raw id stream on the GPU: the step upstream of the
// sampling tables (Sec. 2 trains on a corpus whose words are counted,
// ranked by frequency and cut at a minimum count). It produces what the
// rest of the library expects: ids ranked by frequency (id 0 the most
// frequent word, which the atomic and split update tiers rely on), the
// ranked counts for w2v_build_tables, and the corpus rewritten in ranked
// ids with dropped words marked -1 (the epoch kernels skip such positions
// before forming windows, as the original tool removes them from the
// stream).
//
//   1. counts of the raw ids (ids outside [0, V_raw) are not counted), as
//      sort keys 2^b - 1 - count with b the bit length of T;
//   2. a stable radix sort of the raw ids by key, ascending (radix_sort.hip),
//      i.e. by count, descending, equal counts in increasing raw id order;
//   3. rank r of sorted word s: new id r if its count reaches min_count,
//      else -1; ranked counts out;
//   4. the corpus rewritten through the rank map.
//
// Counting without memory-side atomics (V_raw <= kMaxBins * kBinIds). A
// Zipf stream has a long tail: most distinct ids occur a few times in any
// chunk of the stream, so a per-workgroup cache of counters catches only the
// head and every tail token would cost a global atomic. The ids are split
// instead into P = ceil(V_raw / kBinIds) ranges ("bins") of kBinIds ids,
// small enough for one workgroup to hold a counter for every id of a bin in
// LDS:
//   a. k_vocab_bin: each chunk of kBinChunk tokens is reordered by bin in LDS
//      and written back to a chunk-sized slot of the workspace, each bin's
//      segment padded with -1 to a multiple of 4 ids; the segment offsets of
//      every chunk go to a table (P + 1 int32 per chunk);
//   b. k_vocab_bin_totals / k_vocab_plan: the tokens of each bin, and a plan
//      that cuts every bin's chunks into work units of about kUnitTokens
//      tokens;
//   c. k_vocab_tally: one workgroup per unit counts the unit's segments with
//      LDS atomics and stores its kBinIds counters to a partial table;
//   d. k_vocab_merge: each id's count is the sum of its bin's unit partials,
//      written out as the sort key.
// HBM traffic per token: 4 bytes read and 4 written in (a), 4 read in (c),
// against one 8-byte atomic per tail token before. Larger vocabularies take
// the per-workgroup hash-table count (k_vocab_count_hashed).
#include <hip/hip_runtime.h>

#include "kernel_args.h"
#include "w2v_internal.h"

namespace w2v {

constexpr int kBinShift = 15;
constexpr int32_t kBinIds = 1 << kBinShift;      // ids per bin: 128 KB of LDS counters
constexpr int kMaxBins = 128;                    // V_raw <= 4,194,304
constexpr int kBinThreads = 1024;
constexpr int kBinPerThread = 16;
constexpr int64_t kBinChunk = (int64_t)kBinThreads * kBinPerThread;  // 16,384 tokens
constexpr int64_t kChunkStride = kBinChunk + 4 * kMaxBins;  // slot: chunk + padding
constexpr int64_t kUnitTokens = (int64_t)1 << 20;
constexpr int kTallyThreads = 1024;
constexpr int kTallyBatch = kTallyThreads;      // chunks whose segments a unit reads at once
constexpr int kTallyUnroll = 8;                  // int4 loads in flight per thread
constexpr int kTotalsBlocks = 256;
constexpr int kWave = 64;

namespace {

__device__ __forceinline__ int32_t scan_wave_incl(int32_t x, int lane) {
#pragma unroll
  for (int off = 1; off < kWave; off *= 2) {
    const int32_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  return x;
}

__device__ __forceinline__ int64_t scan_wave_incl64(int64_t x, int lane) {
#pragma unroll
  for (int off = 1; off < kWave; off *= 2) {
    const int64_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  return x;
}

__device__ __forceinline__ uint32_t pad4(uint32_t n) { return (n + 3u) & ~3u; }

}  // namespace

// (a) One workgroup per chunk of kBinChunk tokens. Each token takes its rank
// within its bin from an LDS counter (atomic with return), the bins' padded
// sizes are scanned by one wavefront, the tokens are placed in LDS at
// (segment offset + rank) and the chunk's slot is written with 16-byte
// stores. seg[c][0..P] holds chunk c's segment offsets (seg[c][P] = its
// padded length).
__global__ __launch_bounds__(kBinThreads) void k_vocab_bin(const int32_t* raw, int64_t T,
                                                          int32_t V, int32_t P,
                                                          int32_t* binned, int32_t* seg) {
  __shared__ __align__(16) int32_t stage[kChunkStride];
  __shared__ uint32_t cnt[kMaxBins];
  __shared__ int32_t off[kMaxBins + 1];
  const int tid = threadIdx.x;
  const int64_t c = blockIdx.x;
  const int64_t base = c * kBinChunk;
  if (tid < kMaxBins) cnt[tid] = 0u;
  __syncthreads();
  int32_t x[kBinPerThread];
  uint32_t r[kBinPerThread];
#pragma unroll
  for (int i = 0; i < kBinPerThread; ++i) {
    const int64_t p = base + (int64_t)i * kBinThreads + tid;
    x[i] = p < T ? raw[p] : -1;
  }
#pragma unroll
  for (int i = 0; i < kBinPerThread; ++i) {
    if (x[i] < 0 || x[i] >= V) x[i] = -1;
    r[i] = x[i] >= 0 ? atomicAdd(&cnt[x[i] >> kBinShift], 1u) : 0u;
  }
  __syncthreads();
  if (tid < kWave) {
    const int lane = tid;
    const int b0 = 2 * lane, b1 = 2 * lane + 1;
    const int32_t a0 = b0 < P ? (int32_t)pad4(cnt[b0]) : 0;
    const int32_t a1 = b1 < P ? (int32_t)pad4(cnt[b1]) : 0;
    const int32_t incl = scan_wave_incl(a0 + a1, lane);
    const int32_t ex = incl - a0 - a1;
    if (b0 < P) off[b0] = ex;
    if (b1 < P) off[b1] = ex + a0;
    if (lane == kWave - 1) off[P] = incl;
  }
  __syncthreads();
  int32_t* seg_c = seg + c * (P + 1);
  for (int k = tid; k <= P; k += kBinThreads) seg_c[k] = off[k];
  if (tid < P)  // the padding of each segment
    for (int k = off[tid] + (int)cnt[tid]; k < off[tid + 1]; ++k) stage[k] = -1;
#pragma unroll
  for (int i = 0; i < kBinPerThread; ++i)
    if (x[i] >= 0) stage[off[x[i] >> kBinShift] + (int)r[i]] = x[i];
  __syncthreads();
  const int n4 = off[P] / 4;
  int4* dst = reinterpret_cast<int4*>(binned + c * kChunkStride);
  const int4* src = reinterpret_cast<const int4*>(stage);
  for (int k = tid; k < n4; k += kBinThreads) dst[k] = src[k];
}

// (b) Padded token totals of each bin over a range of chunks: thread (r, b)
// of block g sums bin b over every kTotalsRows-th chunk of the block's range
// (consecutive threads read consecutive table entries), then the rows are
// added in LDS.
constexpr int kTotalsRows = 8;
constexpr int kTotalsThreads = kTotalsRows * kMaxBins;

__global__ __launch_bounds__(kTotalsThreads) void k_vocab_bin_totals(const int32_t* seg,
                                                                     int64_t n_chunks,
                                                                     int32_t P,
                                                                     int64_t* part) {
  __shared__ int64_t acc[kTotalsRows][kMaxBins];
  const int b = threadIdx.x % kMaxBins;
  const int r = threadIdx.x / kMaxBins;
  const int64_t per = (n_chunks + gridDim.x - 1) / gridDim.x;
  const int64_t c0 = (int64_t)blockIdx.x * per;
  const int64_t c1 = c0 + per < n_chunks ? c0 + per : n_chunks;
  int64_t sum = 0;
  if (b < P)
    for (int64_t c = c0 + r; c < c1; c += kTotalsRows)
      sum += seg[c * (P + 1) + b + 1] - seg[c * (P + 1) + b];
  acc[r][b] = sum;
  __syncthreads();
  if (r == 0) {
    for (int k = 1; k < kTotalsRows; ++k) sum += acc[k][b];
    part[(int64_t)blockIdx.x * kMaxBins + b] = sum;
  }
}

// The plan: bin b's chunks go in groups of cg_b consecutive chunks, cg_b =
// max(1, floor(kUnitTokens * n_chunks / total_b)), so a unit holds about
// kUnitTokens tokens; unit_base[b] = units of the bins before b. One
// workgroup: the block totals are added by kTotalsRows rows of threads, the
// units scanned by one wavefront; plan = int64 unit_base[0..P] followed by
// cg[0..P).
__global__ __launch_bounds__(kTotalsThreads) void k_vocab_plan(const int64_t* part,
                                                               int32_t n_part,
                                                               int64_t n_chunks, int32_t P,
                                                               int64_t* plan) {
  __shared__ int64_t acc[kTotalsRows][kMaxBins];
  const int b = threadIdx.x % kMaxBins;
  const int r = threadIdx.x / kMaxBins;
  int64_t sum = 0;
  for (int g = r; g < n_part; g += kTotalsRows) sum += part[(int64_t)g * kMaxBins + b];
  acc[r][b] = sum;
  __syncthreads();
  if (threadIdx.x >= kWave) return;
  const int lane = threadIdx.x;
  int64_t units[2], cg[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int bb = 2 * lane + h;
    int64_t tot = 0;
    for (int k = 0; k < kTotalsRows; ++k) tot += acc[k][bb];
    if (bb >= P) tot = 0;
    cg[h] = tot > 0 ? kUnitTokens * n_chunks / tot : n_chunks;
    if (cg[h] < 1) cg[h] = 1;
    units[h] = tot > 0 ? (n_chunks + cg[h] - 1) / cg[h] : 0;
  }
  const int64_t incl = scan_wave_incl64(units[0] + units[1], lane);
  const int64_t ex = incl - units[0] - units[1];
  int64_t* unit_base = plan;
  int64_t* cgs = plan + (P + 1);
  if (2 * lane < P) {
    unit_base[2 * lane] = ex;
    cgs[2 * lane] = cg[0];
  }
  if (2 * lane + 1 < P) {
    unit_base[2 * lane + 1] = ex + units[0];
    cgs[2 * lane + 1] = cg[1];
  }
  if (lane == kWave - 1) unit_base[P] = incl;
}

// (c) Unit u = (bin b, chunks [c0, c1)): kBinIds LDS counters; the
// segments of up to kTallyBatch chunks at a time are read as one run of
// int4 (a block-wide scan of their lengths; each thread finds the chunk of
// an int4 by binary search over the scan, between the start chunks of the
// two kWindow4-int4 windows around it). Loads are software-pipelined:
// each thread has kTallyUnroll int4 in flight while it adds the previous
// kTallyUnroll, and the next batch's segment bounds are loaded while the
// current batch is counted. One LDS atomic per id, except that the id of the
// first active lane is added once per wavefront with its multiplicity (in a
// Zipf bin most likely its head word, which holds most of its tokens and
// would otherwise serialise the atomic on one address). The counters go to
// partial[u][0..kBinIds). Grid: an upper bound on the number of units; the
// workgroups past the plan's count return at once.
// Start chunks: wstart[k] = the chunk whose run holds int4 k * kWindow4 of
// the batch, so the chunk of int4 v lies in [wstart[v / kWindow4],
// wstart[v / kWindow4 + 1]] (a few chunks) instead of anywhere in the batch.
constexpr int kWindowShift = 10;
constexpr int32_t kWindow4 = 1 << kWindowShift;
constexpr int kMaxWindows = (int)(kTallyBatch * (kChunkStride / 4) / kWindow4) + 2;

struct TallyRun {
  const int32_t* binned;
  const int32_t* pre;
  const int32_t* sbeg;
  const int32_t* wstart;
  int64_t cb;
  int nb;
  int32_t total4;
  int32_t nwin;
};

__device__ __forceinline__ int4 tally_load(const TallyRun& r, int32_t v) {
  if (v >= r.total4) return make_int4(-1, -1, -1, -1);
  const int w = v >> kWindowShift;
  int l = r.wstart[w];       // last chunk with pre[l] <= v
  int h = w + 1 < r.nwin ? r.wstart[w + 1] : r.nb - 1;
  while (l < h) {
    const int m = (l + h + 1) / 2;
    if (r.pre[m] <= v) l = m; else h = m - 1;
  }
  const int4* src =
      reinterpret_cast<const int4*>(r.binned + (r.cb + l) * kChunkStride + r.sbeg[l]);
  return src[v - r.pre[l]];
}

__device__ __forceinline__ void tally_add(uint32_t* cnt, int32_t x, int32_t id0, int lane) {
  const int32_t first = __builtin_amdgcn_readfirstlane(x);
  const unsigned long long m = __ballot(x == first);
  uint32_t val = 1u;
  if (x == first) val = lane == __ffsll(m) - 1 ? (uint32_t)__popcll(m) : 0u;
  if (x >= 0 && val != 0u) atomicAdd(&cnt[x - id0], val);
}

__global__ __launch_bounds__(kTallyThreads) void k_vocab_tally(
    const int32_t* binned, const int32_t* seg, int64_t n_chunks, int32_t P,
    const int64_t* plan, uint32_t* partial) {
  __shared__ uint32_t cnt[kBinIds];
  __shared__ int32_t pre[kTallyBatch + 1];
  __shared__ int32_t sbeg[kTallyBatch];
  __shared__ int32_t wsum[kTallyThreads / kWave];
  __shared__ int32_t wstart[kMaxWindows];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int64_t* unit_base = plan;
  const int64_t* cgs = plan + (P + 1);
  const int64_t u = blockIdx.x;
  if (u >= unit_base[P]) return;
  int lo = 0, hi = P - 1;  // last bin with unit_base[b] <= u
  while (lo < hi) {
    const int mid = (lo + hi + 1) / 2;
    if (unit_base[mid] <= u) lo = mid; else hi = mid - 1;
  }
  const int b = lo;
  const int64_t c0 = (u - unit_base[b]) * cgs[b];
  const int64_t c1 = c0 + cgs[b] < n_chunks ? c0 + cgs[b] : n_chunks;
  const int32_t id0 = b << kBinShift;
  for (int j = tid; j < kBinIds; j += kTallyThreads) cnt[j] = 0u;
  // this thread's segment bounds in the first batch
  int32_t s = 0, e = 0;
  if (c0 + tid < c1) {
    const int32_t* row = seg + (c0 + tid) * (P + 1);
    s = row[b];
    e = row[b + 1];
  }
  for (int64_t cb = c0; cb < c1; cb += kTallyBatch) {
    const int nb = c1 - cb < kTallyBatch ? (int)(c1 - cb) : kTallyBatch;
    __syncthreads();  // counters cleared; the previous batch's pre/sbeg read
    const int32_t len4 = (e - s) / 4;
    int32_t incl = scan_wave_incl(len4, lane);
    if (lane == kWave - 1) wsum[wave] = incl;
    __syncthreads();
    if (wave == 0) {
      const int32_t w = lane < kTallyThreads / kWave ? wsum[lane] : 0;
      const int32_t wi = scan_wave_incl(w, lane);
      if (lane < kTallyThreads / kWave) wsum[lane] = wi - w;
    }
    __syncthreads();
    incl += wsum[wave];
    if (tid < nb) {
      pre[tid + 1] = incl;
      sbeg[tid] = s;
    }
    if (tid == 0) pre[0] = 0;
    // the start chunk of every window of kWindow4 int4 that begins in this
    // thread's run (an empty run starts none)
    if (tid < nb) {
      const int32_t a = incl - len4;
      for (int32_t w = (a + kWindow4 - 1) >> kWindowShift; w * kWindow4 < incl; ++w)
        wstart[w] = tid;
    }
    __syncthreads();
    // the next batch's bounds, in flight while this batch is counted
    s = 0;
    e = 0;
    if (cb + kTallyBatch + tid < c1) {
      const int32_t* row = seg + (cb + kTallyBatch + tid) * (P + 1);
      s = row[b];
      e = row[b + 1];
    }
    const int32_t total4 = pre[nb];
    const TallyRun run{binned, pre,    sbeg, wstart, cb,
                       nb,     total4, (total4 + kWindow4 - 1) >> kWindowShift};
    constexpr int32_t kStep = kTallyThreads * kTallyUnroll;
    int4 q[kTallyUnroll];
#pragma unroll
    for (int t = 0; t < kTallyUnroll; ++t) q[t] = tally_load(run, tid + t * kTallyThreads);
    for (int32_t v0 = tid; v0 < run.total4; v0 += kStep) {
      int4 nq[kTallyUnroll];
#pragma unroll
      for (int t = 0; t < kTallyUnroll; ++t)
        nq[t] = tally_load(run, v0 + kStep + t * kTallyThreads);
#pragma unroll
      for (int t = 0; t < kTallyUnroll; ++t) {
        tally_add(cnt, q[t].x, id0, lane);
        tally_add(cnt, q[t].y, id0, lane);
        tally_add(cnt, q[t].z, id0, lane);
        tally_add(cnt, q[t].w, id0, lane);
      }
#pragma unroll
      for (int t = 0; t < kTallyUnroll; ++t) q[t] = nq[t];
    }
  }
  __syncthreads();
  uint4* dst = reinterpret_cast<uint4*>(partial + u * kBinIds);
  const uint4* srcc = reinterpret_cast<const uint4*>(cnt);
  for (int j = tid; j < kBinIds / 4; j += kTallyThreads) dst[j] = srcc[j];
}

// (d) count of id x = sum of partial[u][x mod kBinIds] over the units of
// its bin, stored as the sort key top - count. The unit range is clipped to
// the partial table (the plan's count never exceeds max_units).
__global__ __launch_bounds__(256) void k_vocab_merge(const uint32_t* partial,
                                                     const int64_t* plan, int64_t max_units,
                                                     int32_t V, unsigned long long top,
                                                     unsigned long long* keys) {
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < V;
       x += (int64_t)gridDim.x * blockDim.x) {
    const int b = (int)(x >> kBinShift);
    const int64_t j = x & (kBinIds - 1);
    const int64_t u1 = plan[b + 1] < max_units ? plan[b + 1] : max_units;
    unsigned long long sum = 0ull;
    for (int64_t u = plan[b]; u < u1; ++u) sum += partial[u * kBinIds + j];
    keys[x] = top - sum;
  }
}

// Larger vocabularies: histogram with per-workgroup LDS tables. Each
// workgroup counts a chunk of kChunkTokens tokens into an open-addressing
// table of kTableSlots (id, count) pairs in LDS (linear probing, at most
// kProbes slots; a token that finds no slot goes to the global count
// directly), then adds every table entry to the global counts and clears the
// table. Head words take a slot early in every chunk, so they cost one
// global atomic per chunk and workgroup; tail words cost one per token.
constexpr int kTableSlots = 16384;  // 128 KB of LDS: one workgroup per CU
constexpr int kProbes = 8;
constexpr int kCountThreads = 1024;
constexpr int64_t kChunkTokens = (int64_t)kCountThreads * 1024;
constexpr int32_t kEmptySlot = -1;

__global__ __launch_bounds__(kCountThreads) void k_vocab_count_hashed(
    const int32_t* raw, int64_t T, int32_t V, unsigned long long* counts) {

  __shared__ int32_t key[kTableSlots];
  __shared__ uint32_t cnt[kTableSlots];
  for (int i = threadIdx.x; i < kTableSlots; i += kCountThreads) {
    key[i] = kEmptySlot;
    cnt[i] = 0u;
  }
  __syncthreads();
  const int64_t n_chunks = (T + kChunkTokens - 1) / kChunkTokens;
  for (int64_t ch = blockIdx.x; ch < n_chunks; ch += gridDim.x) {
    const int64_t end = (ch + 1) * kChunkTokens < T ? (ch + 1) * kChunkTokens : T;
    for (int64_t p = ch * kChunkTokens + threadIdx.x; p < end; p += kCountThreads) {
      const int32_t x = raw[p];
      if (x < 0 || x >= V) continue;
      const uint32_t h = ((uint32_t)x * 2654435761u) >> 18;  // 14 bits
      bool done = false;
      for (int probe = 0; probe < kProbes && !done; ++probe) {
        const int sl = (int)((h + (uint32_t)probe) & (kTableSlots - 1));
        int32_t k = __hip_atomic_load(&key[sl], __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_WORKGROUP);
        if (k == kEmptySlot) {
          k = atomicCAS(&key[sl], kEmptySlot, x);
          if (k == kEmptySlot) k = x;
        }
        if (k == x) {
          atomicAdd(&cnt[sl], 1u);
          done = true;
        }
      }
      if (!done) atomicAdd(&counts[x], 1ull);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < kTableSlots; i += kCountThreads) {
      if (key[i] != kEmptySlot) {
        atomicAdd(&counts[key[i]], (unsigned long long)cnt[i]);
        key[i] = kEmptySlot;
        cnt[i] = 0u;
      }
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void k_vocab_zero(unsigned long long* c,
                                                    int32_t V) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < V;
       i += (int64_t)gridDim.x * blockDim.x)
    c[i] = 0ull;
}

// Sort keys: top - count (top = 2^b - 1 >= every count), so that an
// ascending sort orders the words by count, descending.
__global__ __launch_bounds__(256) void k_vocab_keys(const unsigned long long* counts,
                                                    int32_t V, unsigned long long top,
                                                    unsigned long long* keys) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < V;
       i += (int64_t)gridDim.x * blockDim.x)
    keys[i] = top - counts[i];
}

__global__ __launch_bounds__(256) void k_vocab_rank(
    const unsigned long long* sorted_keys, unsigned long long top,
    const int32_t* sorted_ids, int32_t V, int64_t min_count, int64_t* ranked_counts,
    int32_t* rank_of, int32_t* v_kept) {
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < V;
       r += (int64_t)gridDim.x * blockDim.x) {
    const int64_t c = (int64_t)(top - sorted_keys[r]);
    const bool keep = c >= min_count && c > 0;
    rank_of[sorted_ids[r]] = keep ? (int32_t)r : -1;
    ranked_counts[r] = keep ? c : 0;
    // counts are non-increasing in r: the last kept rank fixes the size
    const int64_t c_next = r + 1 < V ? (int64_t)(top - sorted_keys[r + 1]) : 0;
    const bool next_dropped = r + 1 == V || !(c_next >= min_count && c_next > 0);
    if (keep && next_dropped) *v_kept = (int32_t)(r + 1);
    if (r == 0 && !keep) *v_kept = 0;
  }
}

__device__ __forceinline__ int32_t remap_one(int32_t x, int32_t V,
                                             const int32_t* rank_of) {
  return (x >= 0 && x < V) ? rank_of[x] : -1;
}

// 16-byte loads and stores where raw and out share their alignment, the
// remaining head and tail tokens one by one. Each thread has kRemapUnroll
// loads in flight, then their 4 * kRemapUnroll rank gathers, so that the
// gathers' latency (the rank map does not fit one XCD's L2) overlaps. The
// stream is read and written with non-temporal hints, so that the rank map's
// lines keep their place in L2.
constexpr int kRemapUnroll = 4;

__global__ __launch_bounds__(256) void k_vocab_remap(const int32_t* raw,
                                                     int64_t T, int32_t V,
                                                     const int32_t* rank_of,
                                                     int32_t* out) {
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const bool same = ((uintptr_t)raw & 15u) == ((uintptr_t)out & 15u);
  const int64_t head =
      same ? (int64_t)(((16u - ((uintptr_t)raw & 15u)) & 15u) / 4u) : T;
  const int64_t h = head < T ? head : T;
  for (int64_t p = tid; p < h; p += stride) out[p] = remap_one(raw[p], V, rank_of);
  const int64_t n4 = (T - h) / 4;
  typedef int32_t v4i __attribute__((ext_vector_type(4)));
  const v4i* r4 = reinterpret_cast<const v4i*>(raw + h);
  v4i* o4 = reinterpret_cast<v4i*>(out + h);
  for (int64_t i0 = tid; i0 < n4; i0 += stride * kRemapUnroll) {
    v4i x[kRemapUnroll];
#pragma unroll
    for (int k = 0; k < kRemapUnroll; ++k) {
      const int64_t i = i0 + k * stride;
      x[k] = -1;
      if (i < n4) x[k] = __builtin_nontemporal_load(&r4[i]);
    }
#pragma unroll
    for (int k = 0; k < kRemapUnroll; ++k) {
      x[k].x = remap_one(x[k].x, V, rank_of);
      x[k].y = remap_one(x[k].y, V, rank_of);
      x[k].z = remap_one(x[k].z, V, rank_of);
      x[k].w = remap_one(x[k].w, V, rank_of);
    }
#pragma unroll
    for (int k = 0; k < kRemapUnroll; ++k) {
      const int64_t i = i0 + k * stride;
      if (i < n4) __builtin_nontemporal_store(x[k], &o4[i]);
    }
  }
  for (int64_t p = h + 4 * n4 + tid; p < T; p += stride)
    out[p] = remap_one(raw[p], V, rank_of);
}

static size_t align256(size_t n) { return (n + 255) / 256 * 256; }

size_t vocab_workspace_bytes(int32_t V) {
  // counts, sort keys, sorted keys, sorted ids, sort temporaries
  return 3 * align256(sizeof(unsigned long long) * (size_t)V) +
         align256(sizeof(int32_t) * (size_t)V) +
         align256(radix_sort_temp_bytes(V, sizeof(unsigned long long)));
}

static bool binned_count(int32_t V, int64_t T) {
  return T > 0 && (int64_t)V <= (int64_t)kMaxBins * kBinIds;
}

struct BinLayout {
  int32_t P;
  int64_t n_chunks, max_units;
  size_t binned, seg, part, plan, partial, total;
};

// Workspace of the binned count, after the vocabulary arrays. max_units
// bounds the plan's unit count: a bin with t tokens gets at most 2 t /
// kUnitTokens + 1 units (floor(x) >= x / 2 for x >= 1; one unit per chunk
// when t exceeds kUnitTokens * n_chunks), and the bins hold at most
// n_chunks * kChunkStride tokens together.
static BinLayout bin_layout(int32_t V, int64_t T) {
  BinLayout l{};
  l.P = (int32_t)(((int64_t)V + kBinIds - 1) / kBinIds);
  l.n_chunks = (T + kBinChunk - 1) / kBinChunk;
  l.max_units = 2 * l.n_chunks * kChunkStride / kUnitTokens + l.P;
  l.binned = align256(sizeof(int32_t) * (size_t)(l.n_chunks * kChunkStride));
  l.seg = align256(sizeof(int32_t) * (size_t)(l.n_chunks * (l.P + 1)));
  l.part = align256(sizeof(int64_t) * (size_t)kTotalsBlocks * kMaxBins);
  l.plan = align256(sizeof(int64_t) * (size_t)(2 * l.P + 1));
  l.partial = align256(sizeof(uint32_t) * (size_t)l.max_units * kBinIds);
  l.total = l.binned + l.seg + l.part + l.plan + l.partial;
  return l;
}

size_t vocab_workspace_bytes(int32_t V, int64_t T) {
  return vocab_workspace_bytes(V) + (binned_count(V, T) ? bin_layout(V, T).total : 0);
}

// Bit length of T (every count is at most T), at least 1.
static int count_bits(int64_t T) {
  int b = 1;
  while (b < 63 && (T >> b) != 0) ++b;
  return b;
}

static int vocab_grid(int64_t n) {
  const int64_t b = (n + 255) / 256;
  return (int)(b < 8192 ? (b > 0 ? b : 1) : 8192);
}

hipError_t launch_vocab(const int32_t* raw, int64_t T, int32_t V,
                        int64_t min_count, int64_t* ranked_counts,
                        int32_t* rank_of, int32_t* v_kept, int32_t* corpus_out,
                        void* workspace, hipStream_t s) {
  char* w = (char*)workspace;
  auto* counts = (unsigned long long*)w;
  w += align256(sizeof(unsigned long long) * (size_t)V);
  auto* keys = (unsigned long long*)w;
  w += align256(sizeof(unsigned long long) * (size_t)V);
  auto* sorted_keys = (unsigned long long*)w;
  w += align256(sizeof(unsigned long long) * (size_t)V);
  auto* sorted_ids = (int32_t*)w;
  w += align256(sizeof(int32_t) * (size_t)V);
  void* sort_temp = (void*)w;
  w += align256(radix_sort_temp_bytes(V, sizeof(unsigned long long)));
  const int bits = count_bits(T);
  const unsigned long long top = (bits >= 64) ? ~0ull : ((1ull << bits) - 1ull);

  if (binned_count(V, T)) {
    const BinLayout l = bin_layout(V, T);
    auto* binned = (int32_t*)w;
    w += l.binned;
    auto* seg = (int32_t*)w;
    w += l.seg;
    auto* part = (int64_t*)w;
    w += l.part;
    auto* plan = (int64_t*)w;
    w += l.plan;
    auto* partial = (uint32_t*)w;
    const int n_part = (int)(l.n_chunks < kTotalsBlocks ? l.n_chunks : kTotalsBlocks);
    hipLaunchKernelGGL(k_vocab_bin, dim3((unsigned)l.n_chunks), dim3(kBinThreads), 0, s,
                       raw, T, V, l.P, binned, seg);
    hipLaunchKernelGGL(k_vocab_bin_totals, dim3(n_part), dim3(kTotalsThreads), 0, s,
                       (const int32_t*)seg, l.n_chunks, l.P, part);
    hipLaunchKernelGGL(k_vocab_plan, dim3(1), dim3(kTotalsThreads), 0, s,
                       (const int64_t*)part, n_part, l.n_chunks, l.P, plan);
    hipLaunchKernelGGL(k_vocab_tally, dim3((unsigned)l.max_units), dim3(kTallyThreads), 0,
                       s, (const int32_t*)binned, (const int32_t*)seg, l.n_chunks, l.P,
                       (const int64_t*)plan, partial);
    hipLaunchKernelGGL(k_vocab_merge, dim3(vocab_grid(V)), dim3(256), 0, s,
                       (const uint32_t*)partial, (const int64_t*)plan, l.max_units, V, top,
                       keys);
  } else {
    hipLaunchKernelGGL(k_vocab_zero, dim3(vocab_grid(V)), dim3(256), 0, s, counts, V);
    const int64_t n_chunks = (T + kChunkTokens - 1) / kChunkTokens;
    const int cgrid = (int)(n_chunks < 2048 ? (n_chunks > 0 ? n_chunks : 1) : 2048);
    hipLaunchKernelGGL(k_vocab_count_hashed, dim3(cgrid), dim3(kCountThreads), 0, s, raw,
                       T, V, counts);
    hipLaunchKernelGGL(k_vocab_keys, dim3(vocab_grid(V)), dim3(256), 0, s,
                       (const unsigned long long*)counts, V, top, keys);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // values NULL: the raw ids 0..V-1, so equal counts keep increasing id
  e = radix_sort_pairs((const unsigned long long*)keys, nullptr, sorted_keys, sorted_ids,
                       (int64_t)V, bits, sort_temp, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_vocab_rank, dim3(vocab_grid(V)), dim3(256), 0, s,
                     (const unsigned long long*)sorted_keys, top,
                     (const int32_t*)sorted_ids, V, min_count, ranked_counts,
                     rank_of, v_kept);
  if (corpus_out != nullptr)
    hipLaunchKernelGGL(k_vocab_remap, dim3(vocab_grid(T)), dim3(256), 0, s, raw,
                       T, V, rank_of, corpus_out);
  return hipGetLastError();
}

}  // namespace w2v
