// Achievable-peak microbenchmarks: a streaming read and a streaming write
// of HBM with non-temporal 16-byte accesses, a streaming read of rows in the
// packed SpMM's pattern, and a register loop of fp32 matrix-core
// instructions.  They measure what this GPU sustains, so that
// the per-kernel roofline fractions can be stated against measured peaks as
// well as the datasheet ones.  Nothing on the clustering path calls them.
#include "kkm_internal.h"

namespace kkm {

typedef float peak_f4 __attribute__((ext_vector_type(4)));
typedef float peak_f16v __attribute__((ext_vector_type(16)));

// Workgroup g streams its own contiguous range of 16-byte words (ranges of
// a multiple of 1024 words, the last one shorter), 16 KB per step: thread
// t reads words t, t + 256, t + 512, t + 768 of the step, four loads in
// flight.  The workgroup's sum goes to sums[blockIdx.x], so the loads
// cannot be dropped.
__device__ inline void peak_range(int64_t n4, int64_t& lo, int64_t& hi) {
  const int64_t per = ((n4 + gridDim.x - 1) / gridDim.x + 1023) / 1024 * 1024;
  lo = (int64_t)blockIdx.x * per;
  hi = lo + per < n4 ? lo + per : n4;
}

__global__ __launch_bounds__(256) void peak_read_kernel(const peak_f4* __restrict__ p, int64_t n4,
                                                        float* __restrict__ sums) {
  int64_t lo, hi;
  peak_range(n4, lo, hi);
  float s = 0.f;
  int64_t i = lo + threadIdx.x;
  for (; i + 768 < hi; i += 1024) {
    const peak_f4 a = __builtin_nontemporal_load(p + i);
    const peak_f4 b = __builtin_nontemporal_load(p + i + 256);
    const peak_f4 c = __builtin_nontemporal_load(p + i + 512);
    const peak_f4 d = __builtin_nontemporal_load(p + i + 768);
    s += ((a.x + a.y) + (a.z + a.w)) + ((b.x + b.y) + (b.z + b.w)) + ((c.x + c.y) + (c.z + c.w)) +
         ((d.x + d.y) + (d.z + d.w));
  }
  for (; i < hi; i += 256) {
    const peak_f4 a = __builtin_nontemporal_load(p + i);
    s += (a.x + a.y) + (a.z + a.w);
  }
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  __shared__ float part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) sums[blockIdx.x] = (part[0] + part[1]) + (part[2] + part[3]);
}

__global__ __launch_bounds__(256) void peak_write_kernel(peak_f4* __restrict__ p, int64_t n4, float v) {
  int64_t lo, hi;
  peak_range(n4, lo, hi);
  const peak_f4 w = {v, v, v, v};
  int64_t i = lo + threadIdx.x;
  for (; i + 768 < hi; i += 1024) {
    __builtin_nontemporal_store(w, p + i);
    __builtin_nontemporal_store(w, p + i + 256);
    __builtin_nontemporal_store(w, p + i + 512);
    __builtin_nontemporal_store(w, p + i + 768);
  }
  for (; i < hi; i += 256) __builtin_nontemporal_store(w, p + i);
}

// A streaming read of rows in the pattern of the packed SpMM's loads, without
// its arithmetic.  Workgroup (chunk c, segment s), eight wavefronts, reads
// rows rows[128c .. 128c + 127] of an nrows x ld fp32 matrix over columns
// [s * seg, (s + 1) * seg); wavefront w takes rows 16w .. 16w + 15 of the
// chunk, 128 columns per step: instruction g reads row 2g + h (h = lane / 32)
// at columns 4 (lane % 32) .. +3, two rows of 512 contiguous bytes, and the
// next step's loads are issued before the current step is added, so one
// step is in flight per wavefront.  Row indices are clamped into
// [0, nrows).  sums[c * nseg + s] = the workgroup's fp32 sum of what it read.
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(4))) void peak_rows_kernel(
    const float* __restrict__ A, int64_t nrows, int64_t ld, const int* __restrict__ rows, int nseg, int seg,
    float* __restrict__ sums) {
  const int c = (int)(blockIdx.x / (unsigned)nseg), s = (int)(blockIdx.x % (unsigned)nseg);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, h = lane >> 5, c32 = lane & 31;
  const float* rp[8];
#pragma unroll
  for (int g = 0; g < 8; ++g) {
    int64_t r = rows[(int64_t)c * 128 + w * 16 + 2 * g + h];
    r = r < 0 ? 0 : (r >= nrows ? nrows - 1 : r);
    rp[g] = A + r * ld + (int64_t)s * seg + 4 * c32;
  }
  const int steps = seg / 128;
  peak_f4 buf[8];
#pragma unroll
  for (int g = 0; g < 8; ++g) buf[g] = __builtin_nontemporal_load((const peak_f4*)rp[g]);
  peak_f4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int t = 1; t <= steps; ++t) {
    peak_f4 cur[8];
#pragma unroll
    for (int g = 0; g < 8; ++g) cur[g] = buf[g];
    if (t < steps) {
#pragma unroll
      for (int g = 0; g < 8; ++g) buf[g] = __builtin_nontemporal_load((const peak_f4*)(rp[g] + (int64_t)t * 128));
    }
#pragma unroll
    for (int g = 0; g < 8; ++g) acc += cur[g];
  }
  float v = (acc.x + acc.y) + (acc.z + acc.w);
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  __shared__ float part[8];
  if (lane == 0) part[w] = v;
  __syncthreads();
  if (threadIdx.x == 0)
    sums[blockIdx.x] = ((part[0] + part[1]) + (part[2] + part[3])) + ((part[4] + part[5]) + (part[6] + part[7]));
}

// Four independent accumulation chains of v_mfma_f32_32x32x2_f32 per
// wavefront (32 x 32 x 2 x 2 = 4096 flop each); one float per wavefront out.
__global__ __launch_bounds__(256) void peak_mfma_kernel(int iters, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const float a = 1.f + lane * (1.f / 1024.f), b = 1.f / 4096.f;
  peak_f16v acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  if (lane == 0) out[(int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)] = s;
}

hipError_t launch_peak_read(const void* buf, int64_t bytes, float* sums, hipStream_t s) {
  hipLaunchKernelGGL(peak_read_kernel, dim3(kPeakGrid), dim3(256), 0, s, (const peak_f4*)buf, bytes / 16, sums);
  return hipGetLastError();
}

hipError_t launch_peak_write(void* buf, int64_t bytes, float value, hipStream_t s) {
  hipLaunchKernelGGL(peak_write_kernel, dim3(kPeakGrid), dim3(256), 0, s, (peak_f4*)buf, bytes / 16, value);
  return hipGetLastError();
}

hipError_t launch_peak_rows(const float* buf, int64_t nrows, int64_t ld, const int* rows, int nchunks, int seg,
                            float* sums, hipStream_t s) {
  const int nseg = (int)(ld / seg);
  hipLaunchKernelGGL(peak_rows_kernel, dim3((unsigned)((int64_t)nchunks * nseg)), dim3(512), 0, s, buf, nrows, ld,
                     rows, nseg, seg, sums);
  return hipGetLastError();
}

hipError_t launch_peak_mfma(int iters, float* out, hipStream_t s) {
  hipLaunchKernelGGL(peak_mfma_kernel, dim3(kPeakMfmaGrid), dim3(256), 0, s, iters, out);
  return hipGetLastError();
}

}  // namespace kkm
