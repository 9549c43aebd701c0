// Device helpers for the HogBatch kernels on gfx950 (CDNA4, wave64).
//
//  * Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11): the counter-based
//    generator behind every random decision (subsampling, window shrink,
//    shared negatives), so a draw depends only on (seed, position, epoch).
//  * The linear learning-rate decay, in IEEE fp64.
//  * A wave-wide transposing reduction: 64 per-lane partial sums in, each
//    lane out with the full 64-lane sum of one of them. It pairs values with
//    the gfx950 cross-half swaps (v_permlane32_swap, v_permlane16_swap) and
//    DPP mirrors inside 16-lane rows, halving the live values at every step.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace w2v {

constexpr int kWave = 64;

// ---------------------------------------------------------------- Philox --

struct U64x4 {
  uint64_t v[4];
};

// Philox4x64 with 10 rounds. Constants: the two multipliers and the two Weyl
// key increments published for Philox4x64.
__device__ __forceinline__ U64x4 philox4x64_10(uint64_t c0, uint64_t c1,
                                               uint64_t c2, uint64_t c3,
                                               uint64_t k0, uint64_t k1) {
  constexpr uint64_t kMulA = 0xD2E7470EE14C6C93ull;
  constexpr uint64_t kMulB = 0xCA5A826395121157ull;
  constexpr uint64_t kWeylA = 0x9E3779B97F4A7C15ull;
  constexpr uint64_t kWeylB = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t hiA = __umul64hi(kMulA, c0);
    const uint64_t loA = kMulA * c0;
    const uint64_t hiB = __umul64hi(kMulB, c2);
    const uint64_t loB = kMulB * c2;
    const uint64_t n0 = hiB ^ c1 ^ k0;
    const uint64_t n2 = hiA ^ c3 ^ k1;
    c0 = n0;
    c1 = loB;
    c2 = n2;
    c3 = loA;
    k0 += kWeylA;
    k1 += kWeylB;
  }
  U64x4 out;
  out.v[0] = c0;
  out.v[1] = c1;
  out.v[2] = c2;
  out.v[3] = c3;
  return out;
}

// Block `blk` of the stream of raw position p in epoch e.
__device__ __forceinline__ U64x4 stream_block(uint64_t seed, uint64_t p,
                                              uint64_t e, uint64_t blk) {
  return philox4x64_10(p, e, blk, 0ull, seed, 0ull);
}

// 32-bit word j (0..7) of a block: output j/2, low half for even j.
__device__ __forceinline__ uint32_t block_word(const U64x4& b, int j) {
  const uint64_t v = b.v[j >> 1];
  return (j & 1) ? (uint32_t)(v >> 32) : (uint32_t)v;
}

// floor(r * n / 2^32): maps a 32-bit draw onto [0, n) with integers only.
__device__ __forceinline__ uint64_t scale_draw(uint32_t r, uint64_t n) {
  return ((uint64_t)r * n) >> 32;
}

// ------------------------------------------------------- learning rate --

// alpha0 * max(floor_frac, 1 - (epoch*T + p) / (n_epochs*T)), each operation
// rounded once in IEEE fp64 (no contraction), then rounded to fp32.
__device__ __forceinline__ float decayed_alpha(float alpha0, float floor_frac,
                                               int epoch, int n_epochs,
                                               int64_t T, int64_t p) {
#pragma clang fp contract(off)
  const double done = (double)epoch * (double)T + (double)p;
  const double all = (double)n_epochs * (double)T;
  double frac = 1.0 - done / all;
  const double lo = (double)floor_frac;
  if (frac < lo) frac = lo;
  return (float)((double)alpha0 * frac);
}

// ------------------------------------------------------ wave reductions --

__device__ __forceinline__ float f_swap_sum32(float a, float b) {
  // After the swap, `a` holds (a[0..31], b[0..31]) and `b` holds
  // (a[32..63], b[32..63]); their sum gives lanes 0..31 the total of a over
  // both halves and lanes 32..63 the total of b.
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a),
                                            __float_as_uint(b), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float f_swap_sum16(float a, float b) {
  // Odd 16-lane rows of `a` trade places with even rows of `b`: rows 0 and 2
  // end with a-totals over row pairs (0,1), (2,3); rows 1 and 3 with b-totals.
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a),
                                            __float_as_uint(b), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int kCtrl>
__device__ __forceinline__ float f_dpp(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), kCtrl, 0xF,
                                                 0xF, false));
}

// DPP controls (GFX9 encoding).
constexpr int kDppRowMirror = 0x140;      // lane i <-> 15 - i within 16
constexpr int kDppRowHalfMirror = 0x141;  // lane i <-> 7 - i within 8
constexpr int kDppXor2 = 0x4E;            // quad_perm [2,3,0,1]
constexpr int kDppXor1 = 0xB1;            // quad_perm [1,0,3,2]

// One pairing step inside 16-lane rows: lanes whose `upper` flag is set keep
// (and receive the partner's copy of) b, the others a.
template <int kCtrl>
__device__ __forceinline__ float f_pair_dpp(float a, float b, bool upper) {
  const float keep = upper ? b : a;
  const float send = upper ? a : b;
  return keep + f_dpp<kCtrl>(send);
}

// Transposing reduction of 64 values per lane. On return, lane l holds
// sum over all 64 lanes of v[l]. The partner of each step differs from the
// lane in exactly the bit being split (32, 16, then 8, 4, 2, 1 via mirrors),
// so the six steps together cover every lane once. The steps after the
// first (32 values left):
__device__ __forceinline__ float xpose_tail32(float (&v)[32], int lane) {
#pragma unroll
  for (int j = 0; j < 16; ++j) v[j] = f_swap_sum16(v[j], v[j + 16]);
  const bool b3 = (lane & 8) != 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] = f_pair_dpp<kDppRowMirror>(v[j], v[j + 8], b3);
  const bool b2 = (lane & 4) != 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) v[j] = f_pair_dpp<kDppRowHalfMirror>(v[j], v[j + 4], b2);
  const bool b1 = (lane & 2) != 0;
#pragma unroll
  for (int j = 0; j < 2; ++j) v[j] = f_pair_dpp<kDppXor2>(v[j], v[j + 2], b1);
  const bool b0 = (lane & 1) != 0;
  return f_pair_dpp<kDppXor1>(v[0], v[1], b0);
}

__device__ __forceinline__ float xpose_reduce64(float (&v)[64], int lane) {
  float w[32];
#pragma unroll
  for (int j = 0; j < 32; ++j) w[j] = f_swap_sum32(v[j], v[j + 32]);
  return xpose_tail32(w, lane);
}

// The same reduction with value s produced on demand by value(s) (s a
// compile-time index after unrolling), so that values s and s + 32 are
// formed just before the first step combines them and at most 32 partial
// sums are live at once.
template <class F>
__device__ __forceinline__ float xpose_reduce64_lazy(F&& value, int lane) {
  float w[32];
#pragma unroll
  for (int j = 0; j < 32; ++j) w[j] = f_swap_sum32(value(j), value(j + 32));
  return xpose_tail32(w, lane);
}

// Sum of one float over the wave (every lane gets the total).
__device__ __forceinline__ float wave_sum(float x) {
  x += __shfl_xor(x, 32);
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 8);
  x += __shfl_xor(x, 4);
  x += __shfl_xor(x, 2);
  x += __shfl_xor(x, 1);
  return x;
}

// Minimum of one int over the wave (every lane gets it).
__device__ __forceinline__ int wave_min(int x) {
  x = min(x, __shfl_xor(x, 32));
  x = min(x, __shfl_xor(x, 16));
  x = min(x, __shfl_xor(x, 8));
  x = min(x, __shfl_xor(x, 4));
  x = min(x, __shfl_xor(x, 2));
  x = min(x, __shfl_xor(x, 1));
  return x;
}

// Value of x in lane l (l uniform; a compile-time constant after unrolling
// makes this one v_readlane into a scalar register).
__device__ __forceinline__ float lane_value(float x, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}

__device__ __forceinline__ int uniform_int(int x) {
  return __builtin_amdgcn_readfirstlane(x);
}

__device__ __forceinline__ float uniform_float(float x) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(x)));
}

__device__ __forceinline__ uint64_t lanes_below(int lane) {
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Word 3 of a raw buffer descriptor (data format for untyped 32-bit access).
constexpr int kBufferWord3 = 0x00020000;
// Cache policy of a load that must observe agent-scope atomics of other
// wavefronts (sc1: coherent at device scope).
constexpr int kCoherentLoad = 16;

// Cache policy of the plain (non-atomic) row stores of the Hogwild path:
// sc1 writes through this XCD's L2, so wavefronts on other XCDs (whose
// coherent loads do not see another XCD's L2) read the new row at once.
// Without it a dirty line can stay in one XCD's L2 while other XCDs keep
// reading and rewriting the old row, which overwrites far more updates than
// the minibatch-long read-to-write window of Hogwild would.
constexpr int kCoherentStore = 16;

// Error word of the device (host memory mapped into the device's address
// space): a kernel that skipped work because of an id outside [0, V) stores
// kStatusBadId there; the next library call on the host reports it. The
// store goes to system scope so that the host sees it without a copy.
constexpr int32_t kStatusBadId = 1;

__device__ __forceinline__ void report_bad_ids(int32_t* status, int64_t n_bad) {
  if (status != nullptr && n_bad != 0)
    __hip_atomic_store(status, kStatusBadId, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_SYSTEM);
}

// Coherent (agent-scope) row element load and fp32 atomic add; used for the
// live matrices that other wavefronts update concurrently.
__device__ __forceinline__ float load_live(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void add_live(float* p, float g) {
  unsafeAtomicAdd(p, g);
}

}  // namespace w2v
