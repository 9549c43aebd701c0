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
//   1. histogram of the raw ids (LDS tables per workgroup, then 64-bit
//      atomic counts; ids outside [0, V_raw) are not counted);
//   2. a stable radix sort of the raw ids by count, descending, so equal
//      counts keep increasing raw id order (radix_sort.hip, on the key
//      2^b - 1 - count with b the bit length of T, ascending);
//   3. rank r of sorted word s: new id r if its count reaches min_count,
//      else -1; ranked counts out;
//   4. the corpus rewritten through the rank map.
#include <hip/hip_runtime.h>

#include "kernel_args.h"

namespace w2v {

// Histogram with per-workgroup LDS tables. A Zipf stream sends a large
// share of its tokens to a few words, and global atomics to one address
// queue behind each other at the memory side (1.25 s for 1e9 tokens with one
// atomic per token). Each workgroup therefore counts a chunk of kChunkTokens
// tokens into an open-addressing table of kTableSlots (id, count) pairs in
// LDS (linear probing, at most kProbes slots; a token that finds no slot
// goes to the global count directly), then adds every table entry to the
// global counts and clears the table. Head words take a slot early in
// every chunk, so they cost one global atomic per chunk and workgroup.
constexpr int kTableSlots = 16384;  // 128 KB of LDS: one workgroup per CU
constexpr int kProbes = 8;
constexpr int kCountThreads = 1024;
constexpr int64_t kChunkTokens = (int64_t)kCountThreads * 1024;
constexpr int32_t kEmptySlot = -1;

__global__ __launch_bounds__(kCountThreads) void k_vocab_count(
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

// Four tokens per thread with 16-byte loads and stores where raw and out
// share their alignment; the remaining head and tail tokens one by one.
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
  const int4* r4 = reinterpret_cast<const int4*>(raw + h);
  int4* o4 = reinterpret_cast<int4*>(out + h);
  for (int64_t i = tid; i < n4; i += stride) {
    const int4 x = r4[i];
    o4[i] = make_int4(remap_one(x.x, V, rank_of), remap_one(x.y, V, rank_of),
                      remap_one(x.z, V, rank_of), remap_one(x.w, V, rank_of));
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
  const int bits = count_bits(T);
  const unsigned long long top = (bits >= 64) ? ~0ull : ((1ull << bits) - 1ull);

  hipLaunchKernelGGL(k_vocab_zero, dim3(vocab_grid(V)), dim3(256), 0, s, counts, V);
  const int64_t n_chunks = (T + kChunkTokens - 1) / kChunkTokens;
  const int cgrid = (int)(n_chunks < 2048 ? (n_chunks > 0 ? n_chunks : 1) : 2048);
  hipLaunchKernelGGL(k_vocab_count, dim3(cgrid), dim3(kCountThreads), 0, s, raw, T,
                     V, counts);
  hipLaunchKernelGGL(k_vocab_keys, dim3(vocab_grid(V)), dim3(256), 0, s,
                     (const unsigned long long*)counts, V, top, keys);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // values NULL: the raw ids 0..V-1, so equal counts keep increasing id
  e = radix_sort_pairs((const unsigned long long*)keys, nullptr, sorted_keys, sorted_ids,
                       (int64_t)V, bits, (void*)w, s);
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
