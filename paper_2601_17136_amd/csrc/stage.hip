// Staging of the points and small helpers.
//
// The points X (n x d, fp32, row-major; the paper's P of Section II-B) are
// copied into a zero-padded n_pad x d_pad buffer so the K-build tiles never
// need bounds checks along k; zero columns leave every dot product, and so
// Eq. 1, unchanged.  The squared row norms |x_i|^2 are taken in the same pass
// (the Gaussian kernel's expansion |x|^2 + |y|^2 - 2 x.y needs them).
#include "kkm_internal.h"

namespace kkm {

// One wavefront per row; a fixed shuffle tree makes the norm deterministic.
// maxnrm_bits (zero on entry) receives the largest norm as its IEEE bits
// (non-negative floats order like their bit patterns).
__global__ __launch_bounds__(256) void stage_kernel(const float* __restrict__ X, int64_t n, int d,
                                                    int d_pad, int64_t n_pad,
                                                    float* __restrict__ Xp,
                                                    float* __restrict__ nrm,
                                                    unsigned* __restrict__ maxnrm_bits) {
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= n_pad) return;
  float s = 0.f;
  for (int c = lane; c < d_pad; c += 64) {
    float v = (i < n && c < d) ? X[i * d + c] : 0.f;
    Xp[i * d_pad + c] = v;
    s = fmaf(v, v, s);
  }
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if (lane == 0) {
    nrm[i] = s;
    atomicMax(maxnrm_bits, __float_as_uint(s));
  }
}

hipError_t launch_stage(const float* X, int64_t n, int d, int d_pad, int64_t n_pad, float* Xp,
                        float* nrm, unsigned* maxnrm_bits, hipStream_t s) {
  dim3 grid((unsigned)((n_pad + 3) / 4));
  hipLaunchKernelGGL(stage_kernel, grid, dim3(256), 0, s, X, n, d, d_pad, n_pad, Xp, nrm, maxnrm_bits);
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
