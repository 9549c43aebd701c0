// Snapshot batch of independent HogBatch minibatches on gfx950.
//
// Three launches on the caller's stream:
//   1. zero the fp64 delta buffers (workspace);
//   2. one wavefront per minibatch (persistent grid-stride over the batch):
//      rows are read from the matrices, which stay unchanged during this
//      launch, so every minibatch sees the input matrices; the fp32 updates
//      are added with fp64 atomics into the delta buffers;
//   3. every element with a non-zero delta becomes fp32(M + delta), one
//      rounding per element, so the result does not depend on the order in
//      which the atomics landed beyond fp64 rounding.
#include "kernel_args.h"
#include "sgns_core.h"

namespace w2v {

__global__ __launch_bounds__(256) void k_zero(double* p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    p[i] = 0.0;
}

template <int C, int NMAX, bool kMulti>
__global__ __launch_bounds__(kWave) void k_step(StepArgs a) {
  __shared__ MinibatchLds mb;
  const int lane = threadIdx.x;
  int64_t applied = 0, sum_n = 0, rejected = 0, rows = 0;
  for (int64_t b = blockIdx.x; b < a.B; b += gridDim.x) {
    const int t = a.targets[b];
    int bad = (t < 0 || t >= a.V);
    // input words: present ids compacted in order; -1 = absent
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
    if (any_bad) {
      ++rejected;
    } else if (n > 0) {
      ++applied;
      sum_n += n;
      rows += n_in + n_out;
      const float alpha = a.alpha != nullptr ? a.alpha[b] : a.alpha_scalar;
      float unused = 0.f;
      run_minibatch<C, NMAX, kMulti, false, true>(a.M_in, a.M_out, a.dM_in, a.dM_out,
                                          a.ld, a.D, lane, n_in, n_out, alpha,
                                          0, mb, false, unused);
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

// M = fp32(M + delta) where delta != 0; one wavefront per row.
__global__ __launch_bounds__(256) void k_finalize(float* M, const double* dM,
                                                  int32_t V, int32_t D,
                                                  int64_t ld) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t waves = (int64_t)gridDim.x * (blockDim.x / kWave);
  for (int64_t r = (int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
       r < V; r += waves) {
    for (int col = lane; col < D; col += kWave) {
      const double d = dM[r * ld + col];
      if (d != 0.0) M[r * ld + col] = (float)((double)M[r * ld + col] + d);
    }
  }
}

#define W2V_STEP_SHAPES(X) \
  X(1, 10) X(2, 10) X(3, 10) X(4, 10) X(5, 10) X(6, 10) X(8, 10) X(10, 10) \
  X(1, 16) X(2, 16) X(3, 16) X(4, 16) X(5, 16) X(1, 32) X(2, 32)

using StepKernel = void (*)(StepArgs);

static StepKernel step_kernel_for(int C, int nmax, int K) {
  const bool multi = K + 1 > kWave / nmax;
#define W2V_PICK(c, n) \
  if (C == c && nmax == n) return multi ? k_step<c, n, true> : k_step<c, n, false>;
  W2V_STEP_SHAPES(W2V_PICK)
#undef W2V_PICK
  return nullptr;
}

hipError_t launch_step(int C, int nmax, const StepArgs& a, int grid,
                       hipStream_t s) {
  StepKernel k = step_kernel_for(C, nmax, a.K);
  if (k == nullptr) return hipErrorInvalidValue;
  const int64_t n_delta = (int64_t)a.V * a.ld;
  hipLaunchKernelGGL(k_zero, dim3(4096), dim3(256), 0, s, a.dM_in, n_delta);
  hipLaunchKernelGGL(k_zero, dim3(4096), dim3(256), 0, s, a.dM_out, n_delta);
  hipLaunchKernelGGL(k, dim3(grid), dim3(kWave), 0, s, a);
  const int64_t blocks = ((int64_t)a.V + 3) / 4;
  const int fgrid = (int)(blocks < 65536 ? blocks : 65536);
  hipLaunchKernelGGL(k_finalize, dim3(fgrid), dim3(256), 0, s, a.M_in,
                     (const double*)a.dM_in, a.V, a.D, a.ld);
  hipLaunchKernelGGL(k_finalize, dim3(fgrid), dim3(256), 0, s, a.M_out,
                     (const double*)a.dM_out, a.V, a.D, a.ld);
  return hipGetLastError();
}

}  // namespace w2v
