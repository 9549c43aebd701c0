// Memory-system ceiling for the epoch's access pattern (measurement only;
// not part of the training path). Each wavefront takes `rows` row ids per
// step, the rows of one minibatch, and updates those rows in place the way
// the epoch kernel does: the first `rows - atomic_rows` with a coherent
// load of the row followed by a write-through store of (value + 1), the
// last `atomic_rows` with fp32 atomic adds of 1 performed at the memory
// side. Rows are D floats at stride ld, accessed through range-checked
// buffer descriptors with the epoch kernel's cache policies; the ids come
// from the caller. A step loads all of its plain rows before it stores
// any, so with one wavefront (grid = 1) and distinct rows within each step
// every element of row r ends up increased by exactly the number of times r
// was drawn (a row drawn twice in one step keeps one of the two
// increments); with many wavefronts, concurrent read-modify-writes of one
// row may overwrite each other, as in the epoch's plain tier, while atomic
// rows keep every increment.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kWave = 64;
constexpr int kMaxRows = 16;
constexpr int kCoherent = 16;  // sc1: device-scope coherent load / write-through store

__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(float* row, int n_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(row, (short)0, n_bytes, 0x00020000);
}

template <int C>
__global__ __launch_bounds__(kWave) void k_row_rmw(float* M, int64_t ld, int D,
                                                  const int32_t* ids, int64_t n_steps,
                                                  int rows, int atomic_rows) {
  const int lane = threadIdx.x;
  const int plain = rows - atomic_rows;
  for (int64_t st = blockIdx.x; st < n_steps; st += gridDim.x) {
    const int32_t* sid = ids + st * rows;
    float r[kMaxRows][C];
#pragma unroll
    for (int i = 0; i < kMaxRows; ++i) {
      if (i < plain) {
        const int id = __builtin_amdgcn_readfirstlane(sid[i]);
        const __amdgpu_buffer_rsrc_t rs = row_rsrc(M + (int64_t)id * ld, D * 4);
#pragma unroll
        for (int c = 0; c < C; ++c)
          r[i][c] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
              rs, (lane + kWave * c) * 4, 0, kCoherent));
      }
    }
#pragma unroll
    for (int i = 0; i < kMaxRows; ++i) {
      if (i < rows) {
        const int id = __builtin_amdgcn_readfirstlane(sid[i]);
        const __amdgpu_buffer_rsrc_t rs = row_rsrc(M + (int64_t)id * ld, D * 4);
        if (i < plain) {
#pragma unroll
          for (int c = 0; c < C; ++c)
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(r[i][c] + 1.f), rs,
                                                  (lane + kWave * c) * 4, 0, kCoherent);
        } else {
#pragma unroll
          for (int c = 0; c < C; ++c)
            __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(1.f, rs, (lane + kWave * c) * 4,
                                                            0, 0);
        }
      }
    }
  }
}

}  // namespace

extern "C" {

// M: device float[V][ld]; ids: device int32[n_steps][rows], each in [0, V)
// (not checked on the device: the caller draws them). 1 <= rows <= 16,
// 0 <= atomic_rows <= rows, 1 <= D <= 320, D <= ld. Returns 0, -1 on invalid
// arguments, -2 on a launch error.
int w2v_measure_row_rmw(float* M, int64_t V, int32_t D, int64_t ld, const int32_t* ids,
                        int64_t n_steps, int32_t rows, int32_t atomic_rows, int32_t grid,
                        void* stream) {
  if (M == nullptr || ids == nullptr || V <= 0 || D < 1 || D > 5 * kWave || ld < D ||
      n_steps < 0 || rows < 1 || rows > kMaxRows || atomic_rows < 0 || atomic_rows > rows ||
      grid < 1)
    return -1;
  if (n_steps == 0) return 0;
  const int C = (D + kWave - 1) / kWave;
  hipStream_t s = (hipStream_t)stream;
  switch (C) {
    case 1: hipLaunchKernelGGL(k_row_rmw<1>, dim3(grid), dim3(kWave), 0, s, M, ld, D, ids, n_steps, rows, atomic_rows); break;
    case 2: hipLaunchKernelGGL(k_row_rmw<2>, dim3(grid), dim3(kWave), 0, s, M, ld, D, ids, n_steps, rows, atomic_rows); break;
    case 3: hipLaunchKernelGGL(k_row_rmw<3>, dim3(grid), dim3(kWave), 0, s, M, ld, D, ids, n_steps, rows, atomic_rows); break;
    case 4: hipLaunchKernelGGL(k_row_rmw<4>, dim3(grid), dim3(kWave), 0, s, M, ld, D, ids, n_steps, rows, atomic_rows); break;
    default: hipLaunchKernelGGL(k_row_rmw<5>, dim3(grid), dim3(kWave), 0, s, M, ld, D, ids, n_steps, rows, atomic_rows); break;
  }
  return hipGetLastError() == hipSuccess ? 0 : -2;
}

}  // extern "C"
