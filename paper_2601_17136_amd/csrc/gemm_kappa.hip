// K = kappa(X X^T): the Gram GEMM of Eq. 1 with the kernel function of Eq. 2
// (or the linear / Gaussian kernel) applied in the epilogue.
//
// B = X X^T is symmetric, so only tiles (I, J) with I <= J of the 128 x 128
// tiling are computed; an off-diagonal tile is stored twice, as itself and,
// transposed through LDS, as tile (J, I).  The product runs on the fp32
// matrix cores (v_mfma_f32_32x32x2_f32).  Each 256-thread workgroup owns one
// tile, each wavefront a 64 x 64 quarter of it (2 x 2 MFMA blocks of 32 x 32).
//
// Within a 16-wide k chunk a lane feeds the MFMA from eight consecutive k of
// its row: the half-wave h = lane/32 takes k = 8h .. 8h+7 and step s pairs
// k = s with k = 8 + s.  Summation order over k is free, so this only
// changes which k meet in one instruction, and it lets every lane fetch its
// operands with two 16-byte LDS reads per block.
//
// Gaussian entries are formed as exp(-gamma (|x|^2 + |y|^2 - 2 x.y)).  When
// |x|^2 + |y|^2 is large next to |x - y|^2 this loses digits to cancellation;
// the epilogue estimates the error of each entry and lists the ones whose
// estimate is above a tolerance, and a second kernel recomputes those from
// the coordinate differences.
#include "tile_mma.h"

namespace kkm {

// The t-th tile of the upper triangle in row-major order (row I holds
// J = I .. nt-1), counted from the end so the search runs on the short rows.
__device__ inline void triangle_tile(int64_t t, int64_t nt, int64_t& I, int64_t& J) {
  const int64_t T = nt * (nt + 1) / 2;
  const int64_t u = T - 1 - t;
  int64_t r = (int64_t)((sqrt(8.0 * (double)u + 1.0) - 1.0) * 0.5);
  while ((r + 1) * (r + 2) / 2 <= u) ++r;
  while (r * (r + 1) / 2 > u) --r;
  const int64_t o = u - r * (r + 1) / 2;
  I = nt - 1 - r;
  J = nt - 1 - o;
}

template <int KIND>
__global__ __launch_bounds__(256, 2) void gemm_kappa_kernel(
    const float* __restrict__ Xp, const float* __restrict__ nrm, int64_t n, int d_pad, int64_t ld,
    int64_t nt, int64_t T, KappaParams kp, float* __restrict__ K, float* __restrict__ diagK,
    int2* __restrict__ fix_list, unsigned long long* __restrict__ fix_count, long long fix_cap) {
  __shared__ __attribute__((aligned(16))) float lds[kLdsFloats];

  // Workgroup b runs on XCD b % 8.  Give each XCD a contiguous run of tiles
  // so that concurrent workgroups of one XCD share row block I in its L2.
  const int64_t b = blockIdx.x;
  const int64_t per = T >> 3, rem = T & 7, x = b & 7;
  const int64_t t = x * per + (x < rem ? x : rem) + (b >> 3);
  int64_t I, J;
  triangle_tile(t, nt, I, J);
  const int64_t row0 = I * kTile, col0 = J * kTile;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l32 = lane & 31, h = lane >> 5;

  floatx16 acc[2][2];
  mma_tile(Xp + row0 * d_pad, Xp + col0 * d_pad, d_pad, lds, acc);

  // ---- epilogue: acc[bi][bj][r] is B(i, j) with
  //      i = row0 + wm*64 + bi*32 + 8*(r/4) + 4*h + r%4,  j = col0 + wn*64 + bj*32 + l32
  float nj[2] = {0.f, 0.f};
  if (KIND == GAUSS) {
    nj[0] = nrm[col0 + wn * 64 + l32];
    nj[1] = nrm[col0 + wn * 64 + 32 + l32];
  }
#pragma unroll
  for (int bi = 0; bi < 2; ++bi) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int il = wm * 64 + bi * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
      const int64_t gi = row0 + il;
      const float ni = (KIND == GAUSS) ? nrm[gi] : 0.f;
#pragma unroll
      for (int bj = 0; bj < 2; ++bj) {
        const int jl = wn * 64 + bj * 32 + l32;
        const int64_t gj = col0 + jl;
        float v = kappa<KIND>(acc[bi][bj][r], ni, nj[bj], kp);
        if (I == J && il == jl) {
          if (KIND == GAUSS) v = 1.f;  // exp(0): exact, whatever B(i,i) rounded to
          if (gi < n) diagK[gi] = v;
        }
        if (KIND == GAUSS) {
          const bool f = (gi < gj) && (gj < n) && gauss_needs_fix(v, ni, nj[bj], kp);
          const unsigned long long m = __ballot(f);
          if (m) {
            const int leader = __ffsll((long long)m) - 1;
            unsigned long long base = 0;
            if (lane == leader) base = atomicAdd(fix_count, (unsigned long long)__popcll(m));
            base = __shfl(base, leader, 64);
            if (f) {
              const unsigned long long idx = base + __popcll(m & ((1ull << lane) - 1ull));
              if (idx < (unsigned long long)fix_cap) fix_list[idx] = make_int2((int)gi, (int)gj);
            }
          }
        }
        acc[bi][bj][r] = v;
      }
    }
  }

  // ---- stores, staged through LDS so each instruction writes 256 contiguous bytes
  float* Tw = lds + wave * (32 * 65);
#pragma unroll
  for (int bi = 0; bi < 2; ++bi) {  // tile (I, J): rows i, columns j
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        Tw[(8 * (r >> 2) + 4 * h + (r & 3)) * 65 + bj * 32 + l32] = acc[bi][bj][r];
    __syncthreads();
    const int64_t gj = col0 + wn * 64 + lane;
    for (int rr = 0; rr < 32; ++rr) {
      const int64_t gi = row0 + wm * 64 + bi * 32 + rr;
      if (gi < n && gj < ld) K[gi * ld + gj] = (gj < n) ? Tw[rr * 65 + lane] : 0.f;
    }
    __syncthreads();
  }
  if (I != J) {
#pragma unroll
    for (int bj = 0; bj < 2; ++bj) {  // tile (J, I): rows j, columns i
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          Tw[l32 * 65 + bi * 32 + 8 * (r >> 2) + 4 * h + (r & 3)] = acc[bi][bj][r];
      __syncthreads();
      const int64_t gj = row0 + wm * 64 + lane;  // I < J, so gj < n
      for (int rr = 0; rr < 32; ++rr) {
        const int64_t gi = col0 + wn * 64 + bj * 32 + rr;
        if (gi < n) K[gi * ld + gj] = Tw[rr * 65 + lane];
      }
      __syncthreads();
    }
  }
}

hipError_t launch_gemm_kappa(const float* Xp, const float* nrm, int64_t n, int d_pad, int64_t ld,
                             const KappaParams& kp, float* K, float* diagK, int2* fix_list,
                             unsigned long long* fix_count, long long fix_cap, hipStream_t s) {
  const int64_t nt = (n + kTile - 1) / kTile;
  const int64_t T = nt * (nt + 1) / 2;
  dim3 grid((unsigned)T), block(256);
  switch (kp.kind) {
    case LINEAR:
      hipLaunchKernelGGL(gemm_kappa_kernel<LINEAR>, grid, block, 0, s, Xp, nrm, n, d_pad, ld, nt, T,
                         kp, K, diagK, fix_list, fix_count, fix_cap);
      break;
    case POLY:
      hipLaunchKernelGGL(gemm_kappa_kernel<POLY>, grid, block, 0, s, Xp, nrm, n, d_pad, ld, nt, T,
                         kp, K, diagK, fix_list, fix_count, fix_cap);
      break;
    default:
      hipLaunchKernelGGL(gemm_kappa_kernel<GAUSS>, grid, block, 0, s, Xp, nrm, n, d_pad, ld, nt, T,
                         kp, K, diagK, fix_list, fix_count, fix_cap);
      break;
  }
  return hipGetLastError();
}

// ---- Gaussian fix-up: |x_i - x_j|^2 summed from the coordinate differences.

// 16 lanes per listed pair, float4 steps along k, fixed shuffle tree.
__global__ __launch_bounds__(256) void gauss_fixup_list_kernel(const float* __restrict__ Xp,
                                                               int d_pad, int64_t ld, float neg_g_log2e,
                                                               const int2* __restrict__ list,
                                                               long long count,
                                                               float* __restrict__ K) {
  const int g = threadIdx.x >> 4, gl = threadIdx.x & 15;
  const int nq = d_pad >> 2;
  for (long long p = (long long)blockIdx.x * 16 + g; p < count; p += (long long)gridDim.x * 16) {
    const int2 ij = list[p];
    const float4* xi = (const float4*)(Xp + (int64_t)ij.x * d_pad);
    const float4* xj = (const float4*)(Xp + (int64_t)ij.y * d_pad);
    float s = 0.f;
    for (int c = gl; c < nq; c += 16) {
      const float4 a = xi[c], b = xj[c];
      float dx = a.x - b.x;
      s = fmaf(dx, dx, s);
      dx = a.y - b.y;
      s = fmaf(dx, dx, s);
      dx = a.z - b.z;
      s = fmaf(dx, dx, s);
      dx = a.w - b.w;
      s = fmaf(dx, dx, s);
    }
    s += __shfl_xor(s, 8, 16);
    s += __shfl_xor(s, 4, 16);
    s += __shfl_xor(s, 2, 16);
    s += __shfl_xor(s, 1, 16);
    if (gl == 0) {
      const float v = __builtin_amdgcn_exp2f(neg_g_log2e * s);
      K[(int64_t)ij.x * ld + ij.y] = v;
      K[(int64_t)ij.y * ld + ij.x] = v;
    }
  }
}

hipError_t launch_gauss_fixup_list(const float* Xp, int d_pad, int64_t ld, const KappaParams& kp,
                                   const int2* fix_list, long long count, float* K, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  long long blocks = (count + 15) / 16;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(gauss_fixup_list_kernel, dim3((unsigned)blocks), dim3(256), 0, s, Xp, d_pad,
                     ld, kp.neg_g_log2e, fix_list, count, K);
  return hipGetLastError();
}

// Overflow path: when more entries qualify than the list holds, re-test every
// entry of the upper triangle from the stored K with the epilogue's estimate.
__global__ __launch_bounds__(256) void gauss_fixup_scan_kernel(const float* __restrict__ Xp,
                                                               const float* __restrict__ nrm,
                                                               int64_t n, int d_pad, int64_t ld,
                                                               KappaParams kp,
                                                               float* __restrict__ K) {
  const int64_t i = blockIdx.x;
  const float ni = nrm[i];
  for (int64_t j = i + 1 + threadIdx.x; j < n; j += 256) {
    const float v = K[i * ld + j];
    if (gauss_needs_fix(v, ni, nrm[j], kp)) {
      const float w = gauss_direct(Xp + i * d_pad, Xp + j * d_pad, d_pad, kp);
      K[i * ld + j] = w;
      K[j * ld + i] = w;
    }
  }
}

hipError_t launch_gauss_fixup_scan(const float* Xp, const float* nrm, int64_t n, int d_pad,
                                   int64_t ld, const KappaParams& kp, float* K, hipStream_t s) {
  hipLaunchKernelGGL(gauss_fixup_scan_kernel, dim3((unsigned)n), dim3(256), 0, s, Xp, nrm, n,
                     d_pad, ld, kp, K);
  return hipGetLastError();
}

}  // namespace kkm
