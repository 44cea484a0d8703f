// Staging of the points and small helpers.
//
// The points X (n x d, fp32, row-major; the paper's P of Section II-B) are
// copied into a zero-padded n_pad x d_pad buffer so the K-build tiles never
// need bounds checks along k; zero columns leave every dot product, and so
// Eq. 1, unchanged.  The squared row norms |x_i|^2 are taken in the same pass
// (the Gaussian kernel's expansion |x|^2 + |y|^2 - 2 x.y needs them).
#include "kkm_internal.h"

namespace kkm {

// Each wavefront stages kStageRows rows at once (their loads in flight
// together); per row, lane l sums the squares of columns l, l+64, ... in order
// and a fixed shuffle tree adds the lanes, so the norm is deterministic.
// maxnrm_bits (zero on entry) receives the largest norm as its IEEE bits
// (non-negative floats order like their bit patterns); a workgroup takes the
// max of its rows in LDS and updates the word only when its max is larger than
// what the word already holds.  A stale read only costs a redundant atomic.
constexpr int kStageRows = 4;
constexpr int kStageWaves = 4;

__global__ __launch_bounds__(64 * kStageWaves) void stage_kernel(const float* __restrict__ X, int64_t n,
                                                                 int d, int d_pad, int64_t n_pad,
                                                                 float* __restrict__ Xp,
                                                                 float* __restrict__ nrm,
                                                                 unsigned* __restrict__ maxnrm_bits) {
  __shared__ float wmax[kStageWaves];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t i0 = ((int64_t)blockIdx.x * kStageWaves + w) * kStageRows;
  float s[kStageRows];
#pragma unroll
  for (int r = 0; r < kStageRows; ++r) s[r] = 0.f;
  for (int c = lane; c < d_pad; c += 64) {
    float v[kStageRows];
#pragma unroll
    for (int r = 0; r < kStageRows; ++r) {
      const int64_t i = i0 + r;
      v[r] = (i < n && c < d) ? X[i * d + c] : 0.f;
    }
#pragma unroll
    for (int r = 0; r < kStageRows; ++r) {
      const int64_t i = i0 + r;
      if (i < n_pad) Xp[i * d_pad + c] = v[r];
      s[r] = fmaf(v[r], v[r], s[r]);
    }
  }
  float m = 0.f;
#pragma unroll
  for (int r = 0; r < kStageRows; ++r) {
    for (int off = 32; off > 0; off >>= 1) s[r] += __shfl_xor(s[r], off, 64);
    if (lane == r && i0 + r < n_pad) nrm[i0 + r] = s[r];
    m = fmaxf(m, s[r]);
  }
  if (lane == 0) wmax[w] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int q = 1; q < kStageWaves; ++q) m = fmaxf(m, wmax[q]);
    const unsigned bits = __float_as_uint(m);
    if (__hip_atomic_load(maxnrm_bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < bits)
      atomicMax(maxnrm_bits, bits);
  }
}

hipError_t launch_stage(const float* X, int64_t n, int d, int d_pad, int64_t n_pad, float* Xp,
                        float* nrm, unsigned* maxnrm_bits, hipStream_t s) {
  const int64_t rows = (int64_t)kStageRows * kStageWaves;
  dim3 grid((unsigned)((n_pad + rows - 1) / rows));
  hipLaunchKernelGGL(stage_kernel, grid, dim3(64 * kStageWaves), 0, s, X, n, d, d_pad, n_pad, Xp, nrm,
                     maxnrm_bits);
  return hipGetLastError();
}

// tr K in fp64 with a fixed reduction order (one workgroup).
__global__ __launch_bounds__(1024) void trace_kernel(const float* __restrict__ diagK, int64_t n,
                                                     double* __restrict__ out) {
  __shared__ double part[1024];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += 1024) s += (double)diagK[i];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = part[0];
}

hipError_t launch_trace(const float* diagK, int64_t n, double* trK, hipStream_t s) {
  hipLaunchKernelGGL(trace_kernel, dim3(1), dim3(1024), 0, s, diagK, n, trK);
  return hipGetLastError();
}

__global__ void fill_kernel(float* __restrict__ p, int64_t count, float v) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) p[i] = v;
}

hipError_t launch_fill_diag(float* diagK, int64_t n, float v, hipStream_t s) {
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, diagK, n, v);
  return hipGetLastError();
}

__global__ void zero_ints_kernel(int* __restrict__ p, int64_t count) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) p[i] = 0;
}

// A fill kernel rather than hipMemsetAsync, so a captured graph replays it safely.
hipError_t launch_zero_ints(int* p, int64_t count, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_ints_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, p,
                     count);
  return hipGetLastError();
}

}  // namespace kkm
