// Stable least-significant-digit radix sort of (key, value) pairs on gfx950,
// written for the library's two sorts: the snapshot batch's staging rows by
// matrix row (keys < 2V + 1, values = staging indices) and the vocabulary's
// words by count (keys = max count - count, values = raw ids).
//
// Each pass sorts by one 6-bit digit, so one wavefront's 64 lanes hold the
// 64 digit counters. The input is cut into tiles of kRadixGroups x 64
// elements, one wavefront per tile:
//   1. k_radix_hist: the tile's count of every digit, written digit-major
//      (hist[digit][tile]);
//   2. k_radix_scan: one wavefront per digit turns its row into exclusive
//      prefix sums over the tiles and records the digit's total;
//   3. k_radix_scatter: each tile's wavefront scans the 64 totals (the
//      digit's base), then sends the tile's elements out in input order,
//      each to base + row prefix + its rank, its digit's next position.
// Within a group of 64 elements the lanes holding the same digit are found
// with six ballots (one per digit bit); a lane's rank among them is the
// number of such lanes below it. Elements of equal digit therefore keep
// their input order, inside a tile and across tiles, so every pass is
// stable and so is the sort.
#include <hip/hip_runtime.h>

#include "device_common.h"
#include "kernel_args.h"

namespace w2v {

constexpr int kRadixBits = 6;
constexpr int kRadixDigits = 1 << kRadixBits;  // = kWave
constexpr int kRadixGroups = 16;                // groups of 64 per tile
constexpr int64_t kRadixTile = (int64_t)kWave * kRadixGroups;
static_assert(kRadixDigits == kWave, "one digit counter per lane");

// Lanes whose element is valid and has digit d (this lane's digit).
__device__ __forceinline__ uint64_t same_digit(int d, bool valid) {
  uint64_t m = __ballot(valid);
#pragma unroll
  for (int b = 0; b < kRadixBits; ++b) {
    const bool bit = ((d >> b) & 1) != 0;
    const uint64_t set = __ballot(valid && bit);
    m &= bit ? set : ~set;
  }
  return m;
}

// The tile's keys (and values), all loaded before any is used so that the
// loads overlap: element g * 64 + lane of tile `tile` in k[g] (0 past n).
template <class Key>
__device__ __forceinline__ void load_tile(const Key* keys, const int32_t* vals,
                                          int64_t n, int64_t tile, int lane,
                                          Key (&k)[kRadixGroups],
                                          int32_t (&v)[kRadixGroups]) {
#pragma unroll
  for (int g = 0; g < kRadixGroups; ++g) {
    const int64_t i = tile * kRadixTile + (int64_t)g * kWave + lane;
    const int64_t ic = i < n ? i : n - 1;  // in range, not used past n
    k[g] = keys[ic];
    v[g] = vals != nullptr ? vals[ic] : (int32_t)i;
  }
}

template <class Key>
__global__ __launch_bounds__(kWave) void k_radix_hist(const Key* keys, int64_t n,
                                                      int shift, int32_t* hist,
                                                      int64_t n_tiles) {
  __shared__ int32_t cnt[kRadixDigits];
  const int lane = threadIdx.x;
  for (int64_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
    cnt[lane] = 0;
    Key kk[kRadixGroups];
    int32_t unused[kRadixGroups];
    load_tile<Key>(keys, nullptr, n, tile, lane, kk, unused);
    __syncthreads();
#pragma unroll
    for (int g = 0; g < kRadixGroups; ++g) {
      const int64_t i = tile * kRadixTile + (int64_t)g * kWave + lane;
      const bool valid = i < n;
      const int d = valid ? (int)((kk[g] >> shift) & (kRadixDigits - 1)) : 0;
      const uint64_t m = same_digit(d, valid);
      // the lowest lane of each digit adds the group's count of it
      if (valid && (m & lanes_below(lane)) == 0ull) cnt[d] += __popcll(m);
      __syncthreads();
    }
    hist[(int64_t)lane * n_tiles + tile] = cnt[lane];
    __syncthreads();
  }
}

// Per-digit exclusive prefix sums over the tiles, in place, of the
// digit-major table h[d][t] (d < 64 digits, t < n_tiles), and the digit
// totals: one wavefront per digit row. A row goes by in spans of 64 x
// kScanUnroll entries, lane j holding kScanUnroll consecutive ones: each
// lane prefixes its own entries and one wave-wide scan of the lane totals
// per span joins them. The scatter adds each digit's base (the totals of
// the smaller digits). All values fit in int32 (they are counts below
// n < 2^31).
constexpr int kScanUnroll = 16;

__device__ __forceinline__ int32_t wave_inclusive_scan(int32_t x, int lane) {
#pragma unroll
  for (int off = 1; off < kWave; off *= 2) {
    const int32_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  return x;
}

// Range-checked access to the rest of one digit row (n entries from row):
// loads past the end return 0 and stores past it are dropped, so a span's
// loads carry no branch and stay in flight together.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t scan_row(int32_t* row, int64_t n) {
  return __builtin_amdgcn_make_buffer_rsrc(row, (short)0, (int)(n * 4), kBufferWord3);
}

__global__ __launch_bounds__(kWave) void k_radix_scan(int32_t* h, int64_t n_tiles,
                                                      int32_t* totals) {
  const int lane = threadIdx.x;
  constexpr int64_t kSpanEntries = (int64_t)kWave * kScanUnroll;
  for (int d = blockIdx.x; d < kRadixDigits; d += gridDim.x) {
    int32_t* row = h + (int64_t)d * n_tiles;
    int32_t carry = 0;
    for (int64_t b = 0; b < n_tiles; b += kSpanEntries) {
      const __amdgpu_buffer_rsrc_t rs = scan_row(row + b, n_tiles - b);
      int32_t v[kScanUnroll];
#pragma unroll
      for (int u = 0; u < kScanUnroll; ++u)
        v[u] = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(
            rs, (lane * kScanUnroll + u) * 4, 0, 0);
      int32_t own = 0;  // this lane's entries before entry u
      int32_t excl[kScanUnroll];
#pragma unroll
      for (int u = 0; u < kScanUnroll; ++u) {
        excl[u] = own;
        own += v[u];
      }
      const int32_t incl = wave_inclusive_scan(own, lane);
      const int32_t first = carry + incl - own;
#pragma unroll
      for (int u = 0; u < kScanUnroll; ++u)
        __builtin_amdgcn_raw_buffer_store_b32((uint32_t)(first + excl[u]), rs,
                                              (lane * kScanUnroll + u) * 4, 0, 0);
      carry += __shfl(incl, kWave - 1);
    }
    if (lane == 0) totals[d] = carry;
  }
}

template <class Key>
__global__ __launch_bounds__(kWave) void k_radix_scatter(
    const Key* keys_in, const int32_t* vals_in, int64_t n, int shift,
    const int32_t* hist, const int32_t* totals, int64_t n_tiles, Key* keys_out,
    int32_t* vals_out) {
  __shared__ int32_t next[kRadixDigits];
  const int lane = threadIdx.x;
  // first output position of digit `lane`: the totals of the smaller digits
  const int32_t tot = totals[lane];
  const int32_t base = wave_inclusive_scan(tot, lane) - tot;
  for (int64_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
    next[lane] = base + hist[(int64_t)lane * n_tiles + tile];
    Key kk[kRadixGroups];
    int32_t vv[kRadixGroups];
    load_tile<Key>(keys_in, vals_in, n, tile, lane, kk, vv);
    __syncthreads();
#pragma unroll
    for (int g = 0; g < kRadixGroups; ++g) {
      const int64_t i = tile * kRadixTile + (int64_t)g * kWave + lane;
      const bool valid = i < n;
      const Key k = kk[g];
      const int32_t v = vv[g];
      const int d = (int)((k >> shift) & (kRadixDigits - 1));
      const uint64_t m = same_digit(d, valid);
      const int rank = __popcll(m & lanes_below(lane));
      const int32_t pos = valid ? next[d] + rank : 0;
      __syncthreads();
      // positions lie in [0, n) by construction; the test keeps a fault out
      // of reach should the tables ever disagree
      if (valid && pos >= 0 && (int64_t)pos < n) {
        keys_out[pos] = k;
        vals_out[pos] = v;
        // the highest lane of each digit moves the digit's next position
        if (rank == __popcll(m) - 1) next[d] = pos + 1;
      }
      __syncthreads();
    }
  }
}

static size_t radix_align(size_t x) { return (x + 255) / 256 * 256; }

static int64_t radix_tiles(int64_t n) { return (n + kRadixTile - 1) / kRadixTile; }

size_t radix_sort_temp_bytes(int64_t n, size_t key_bytes) {
  if (n <= 0) return 0;
  return radix_align(sizeof(int32_t) * (size_t)kRadixDigits * (size_t)radix_tiles(n)) +
         radix_align(sizeof(int32_t) * (size_t)kRadixDigits) +
         radix_align(key_bytes * (size_t)n) + radix_align(sizeof(int32_t) * (size_t)n);
}

template <class Key>
static hipError_t radix_sort_impl(const Key* keys_in, const int32_t* vals_in,
                                  Key* keys_out, int32_t* vals_out, int64_t n,
                                  int bits, void* temp, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (n > (int64_t)INT32_MAX || bits < 1 || bits > (int)(8 * sizeof(Key)))
    return hipErrorInvalidValue;
  const int64_t n_tiles = radix_tiles(n);
  char* w = (char*)temp;
  int32_t* hist = (int32_t*)w;
  w += radix_align(sizeof(int32_t) * (size_t)kRadixDigits * (size_t)n_tiles);
  int32_t* totals = (int32_t*)w;
  w += radix_align(sizeof(int32_t) * (size_t)kRadixDigits);
  Key* k_tmp = (Key*)w;
  w += radix_align(sizeof(Key) * (size_t)n);
  int32_t* v_tmp = (int32_t*)w;
  const int passes = (bits + kRadixBits - 1) / kRadixBits;
  const int grid = (int)(n_tiles < 65536 ? n_tiles : 65536);
  const Key* ks = keys_in;
  const int32_t* vs = vals_in;
  for (int p = 0; p < passes; ++p) {
    // the last pass writes the caller's output
    const bool to_out = ((passes - 1 - p) % 2) == 0;
    Key* kd = to_out ? keys_out : k_tmp;
    int32_t* vd = to_out ? vals_out : v_tmp;
    const int shift = p * kRadixBits;
    hipLaunchKernelGGL(k_radix_hist<Key>, dim3(grid), dim3(kWave), 0, s, ks, n, shift,
                       hist, n_tiles);
    hipLaunchKernelGGL(k_radix_scan, dim3(kRadixDigits), dim3(kWave), 0, s, hist,
                       n_tiles, totals);
    hipLaunchKernelGGL(k_radix_scatter<Key>, dim3(grid), dim3(kWave), 0, s, ks, vs, n,
                       shift, (const int32_t*)hist, (const int32_t*)totals, n_tiles,
                       kd, vd);
    ks = kd;
    vs = vd;
  }
  return hipGetLastError();
}

hipError_t radix_sort_pairs(const uint32_t* keys_in, const int32_t* vals_in,
                            uint32_t* keys_out, int32_t* vals_out, int64_t n,
                            int bits, void* temp, hipStream_t s) {
  return radix_sort_impl<uint32_t>(keys_in, vals_in, keys_out, vals_out, n, bits, temp, s);
}

hipError_t radix_sort_pairs(const unsigned long long* keys_in, const int32_t* vals_in,
                            unsigned long long* keys_out, int32_t* vals_out, int64_t n,
                            int bits, void* temp, hipStream_t s) {
  return radix_sort_impl<unsigned long long>(keys_in, vals_in, keys_out, vals_out, n,
                                             bits, temp, s);
}

}  // namespace w2v
