// On-the-fly updates: K is never stored.  Every update recomputes the tiles
// of K = kappa(X X^T) on the fp32 matrix cores and folds them straight into
// E = K V^T, the paper's single-GPU sliding-window baseline (Section VI-D)
// done at tile granularity, with V one-hot instead of dense.
//
// The points are first gathered into cluster-sorted order (the same stable
// sort the resident path uses), so along a row of K the columns of one
// cluster form one contiguous run.  A workgroup owns a block of 128 sorted
// rows and sweeps a segment of 128-column tiles in order.  Each lane keeps,
// for each of its 32 rows, the running sum of its own columns' entries;
// when the sweep leaves a cluster the lanes' sums are reduced across the
// workgroup in a fixed order and written as that cluster's partial for the
// segment.  A second kernel adds the segments in order.  E comes out in
// sorted row order; the assign kernel reads it through the inverse
// permutation.
#include "tile_mma.h"

namespace kkm {

// Xs[p] = Xp[perm[p]], nrm_s[p] = nrm[perm[p]], cs[p] = cl[perm[p]] for p < n;
// rows n .. n_pad-1 zero with cs = -1.  One wavefront per row.
__global__ __launch_bounds__(256) void gather_sorted_kernel(const float* __restrict__ Xp,
                                                            const float* __restrict__ nrm,
                                                            const int* __restrict__ perm,
                                                            const int* __restrict__ cl, int64_t n,
                                                            int64_t n_pad, int d_pad, int k,
                                                            float* __restrict__ Xs,
                                                            float* __restrict__ nrm_s,
                                                            int* __restrict__ cs) {
  const int lane = threadIdx.x & 63;
  const int64_t p = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (p >= n_pad) return;
  const int64_t src = p < n ? (int64_t)perm[p] : -1;
  for (int c = lane * 4; c < d_pad; c += 256) {
    const float4 v = src >= 0 ? *(const float4*)(Xp + src * d_pad + c) : make_float4(0.f, 0.f, 0.f, 0.f);
    *(float4*)(Xs + p * d_pad + c) = v;
  }
  if (lane == 0) {
    nrm_s[p] = src >= 0 ? nrm[src] : 0.f;
    const int c = src >= 0 ? cl[src] : -1;
    cs[p] = src < 0 ? -1 : (c < 0 ? 0 : (c >= k ? k - 1 : c));
  }
}

// diag K from the squared norms: LINEAR |x|^2, POLY (gamma |x|^2 + c)^p, GAUSS 1.
template <int KIND>
__global__ void diag_from_norms_kernel(const float* __restrict__ nrm, int64_t n, KappaParams kp,
                                       float* __restrict__ diagK) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  diagK[i] = KIND == GAUSS ? 1.f : kappa<KIND>(nrm[i], 0.f, 0.f, kp);
}

// One 128 x 128 tile of K from its B tile (acc), rows at row0 and columns at
// col0 of the staged points Y (n_pad x d_pad, norms ny): kappa applied, the
// Gaussian diagonal set to exactly 1, columns >= n zeroed, and Gaussian
// entries flagged as cancellation-prone recomputed from the differences.
template <int KIND>
__device__ inline void kappa_tile(floatx16 acc[2][2], const float* __restrict__ Y,
                                  const float* __restrict__ ny, int64_t n, int d_pad,
                                  int64_t row0, int64_t col0, const KappaParams& kp, bool may_fix) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1, l32 = lane & 31, h = lane >> 5;
  float nj[2] = {0.f, 0.f};
  if (KIND == GAUSS) {
    nj[0] = ny[col0 + wn * 64 + l32];
    nj[1] = ny[col0 + wn * 64 + 32 + l32];
  }
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t gi = row0 + wm * 64 + bi * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
      const float ni = (KIND == GAUSS) ? ny[gi] : 0.f;
#pragma unroll
      for (int bj = 0; bj < 2; ++bj) {
        const int64_t gj = col0 + wn * 64 + bj * 32 + l32;
        float v = kappa<KIND>(acc[bi][bj][r], ni, nj[bj], kp);
        if (KIND == GAUSS) {
          if (gi == gj) v = 1.f;
          else if (may_fix && gj < n && gi < n && gauss_needs_fix(v, ni, nj[bj], kp))
            v = gauss_direct(Y + gi * d_pad, Y + gj * d_pad, d_pad, kp);
        }
        acc[bi][bj][r] = gj < n ? v : 0.f;
      }
    }
}

// Segment bounds: segment s of nseg covers column tiles [jt0, jt1).
__device__ __host__ inline int seg_begin(int s, int nt, int nseg) { return (int)((int64_t)s * nt / nseg); }

// Whether any Gaussian entry may need the fix-up, from the largest norm.
__device__ inline bool any_fix(const unsigned* maxnrm_bits, const KappaParams& kp) {
  const float m = __uint_as_float(*maxnrm_bits);
  return kp.kind == GAUSS && gauss_needs_fix(1.f, m, m, kp);
}

template <int KIND>
__global__ __launch_bounds__(256, 2) void onthefly_kernel(const float* __restrict__ Xs,
                                                          const float* __restrict__ nrm_s,
                                                          const int* __restrict__ cs,
                                                          const unsigned* __restrict__ maxnrm_bits,
                                                          int64_t n, int d_pad, int64_t ld, int nt,
                                                          int nseg, int k, KappaParams kp,
                                                          float* __restrict__ Epart) {
  __shared__ __attribute__((aligned(16))) float lds[kLdsFloats];
  const bool may_fix = any_fix(maxnrm_bits, kp);
  __shared__ float red[2][2][64];
  // Workgroup b runs on XCD b % 8; consecutive logical indices share a
  // segment, so the workgroups of one XCD sweep the same column tiles.
  const int64_t T = (int64_t)nt * nseg;
  const int64_t b = blockIdx.x;
  const int64_t per = T >> 3, rem = T & 7, x = b & 7;
  const int64_t t = x * per + (x < rem ? x : rem) + (b >> 3);
  const int I = (int)(t % nt), s = (int)(t / nt);
  const int jt0 = seg_begin(s, nt, nseg), jt1 = seg_begin(s + 1, nt, nseg);
  const int64_t row0 = (int64_t)I * kTile;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, l32 = lane & 31, h = lane >> 5;

  float rowacc[2][16];
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int r = 0; r < 16; ++r) rowacc[bi][r] = 0.f;

  // Reduce the lanes' running sums over the 128 columns of each row and write
  // them as cluster c's partial for this segment; fixed order throughout.
  auto flush = [&](int c) {
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float v = rowacc[bi][r];
        v += __shfl_xor(v, 16, 64);
        v += __shfl_xor(v, 8, 64);
        v += __shfl_xor(v, 4, 64);
        v += __shfl_xor(v, 2, 64);
        v += __shfl_xor(v, 1, 64);
        if (l32 == 0) red[wm][wn][bi * 32 + 8 * (r >> 2) + 4 * h + (r & 3)] = v;
        rowacc[bi][r] = 0.f;
      }
    __syncthreads();
    if (wn == 0) {
      const int64_t gi = row0 + wm * 64 + lane;
      if (gi < n) Epart[((int64_t)s * k + c) * ld + gi] = red[wm][0][lane] + red[wm][1][lane];
    }
    __syncthreads();
  };

  int cur = cs[(int64_t)jt0 * kTile];
  floatx16 acc[2][2];
  for (int J = jt0; J < jt1; ++J) {
    const int64_t col0 = (int64_t)J * kTile;
    mma_tile(Xs + row0 * d_pad, Xs + col0 * d_pad, d_pad, lds, acc);
    kappa_tile<KIND>(acc, Xs, nrm_s, n, d_pad, row0, col0, kp, may_fix);
    const int64_t last = (col0 + kTile - 1 < n) ? col0 + kTile - 1 : n - 1;
    const int cf = cs[col0], cl_last = cs[last];
    if (cf == cur && cl_last == cur) {
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int r = 0; r < 16; ++r) rowacc[bi][r] += acc[bi][0][r] + acc[bi][1][r];
    } else {
      const int64_t q0 = col0 + wn * 64 + l32, q1 = q0 + 32;
      const int c0 = q0 < n ? cs[q0] : -1, c1 = q1 < n ? cs[q1] : -1;
      for (int c = cf; c <= cl_last; ++c) {
        if (c != cur) {
          flush(cur);
          cur = c;
        }
#pragma unroll
        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            rowacc[bi][r] += (c0 == c ? acc[bi][0][r] : 0.f) + (c1 == c ? acc[bi][1][r] : 0.f);
      }
    }
  }
  flush(cur);
}

// Workgroup (stripe, j): E^T_sorted(j, stripe) = sum over the segments that
// overlap cluster j's sorted range, in segment order; plus the stripe's part
// of sum_{p in L_j} E(p, j) in fp64 (sorted positions: cs[p] == j).
__global__ __launch_bounds__(256) void onthefly_reduce_kernel(IterBufs b,
                                                              const float* __restrict__ Epart,
                                                              const int* __restrict__ cs, int nt,
                                                              int nseg) {
  const int ns = b.nstripes;
  const int stripe = (int)(blockIdx.x % (unsigned)ns);
  const int j = (int)(blockIdx.x / (unsigned)ns);
  const int lo = b.off[j], hi = b.off[j + 1];
  if (lo == hi) return;
  const int tid = threadIdx.x;
  __shared__ double red[4];
  typedef float f4 __attribute__((ext_vector_type(4)));
  const int64_t ld = b.ld;
  const int64_t col = (int64_t)stripe * kStripe + tid * 4;
  double zs = 0.0;
  if (col < ld) {
    f4 e = {0.f, 0.f, 0.f, 0.f};
    bool first = true;
    for (int s = 0; s < nseg; ++s) {
      const int64_t c0 = (int64_t)seg_begin(s, nt, nseg) * kTile;
      const int64_t c1 = (int64_t)seg_begin(s + 1, nt, nseg) * kTile;
      if (c0 < hi && lo < c1) {
        const f4 v = *(const f4*)(Epart + ((int64_t)s * b.k + j) * ld + col);
        e = first ? v : e + v;
        first = false;
      }
    }
    *(f4*)(b.Et + (int64_t)j * ld + col) = e;
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (col + c < b.n && cs[col + c] == j) zs += (double)e[c];
  }
  for (int off = 32; off > 0; off >>= 1) zs += __shfl_xor(zs, off, 64);
  if ((tid & 63) == 0) red[tid >> 6] = zs;
  __syncthreads();
  if (tid == 0) b.zpart[(int64_t)j * ns + stripe] = (red[0] + red[1]) + (red[2] + red[3]);
}

// Rows [r0, r1) of K in original order into out ((r1 - r0) x n), by the same
// tile mainloop and kappa epilogue the on-the-fly sweep uses.
template <int KIND>
__global__ __launch_bounds__(256, 2) void kernel_rows_kernel(const float* __restrict__ Xp,
                                                             const float* __restrict__ nrm,
                                                             const unsigned* __restrict__ maxnrm_bits,
                                                             int64_t n, int d_pad, int64_t R0,
                                                             int64_t r0, int64_t r1, int nt,
                                                             KappaParams kp, float* __restrict__ out) {
  __shared__ __attribute__((aligned(16))) float lds[kLdsFloats];
  const bool may_fix = any_fix(maxnrm_bits, kp);
  const int J = (int)(blockIdx.x % (unsigned)nt), I = (int)(blockIdx.x / (unsigned)nt);
  const int64_t row0 = R0 + (int64_t)I * kTile, col0 = (int64_t)J * kTile;
  floatx16 acc[2][2];
  mma_tile(Xp + row0 * d_pad, Xp + col0 * d_pad, d_pad, lds, acc);
  kappa_tile<KIND>(acc, Xp, nrm, n, d_pad, row0, col0, kp, may_fix);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1, l32 = lane & 31, h = lane >> 5;
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t gi = row0 + wm * 64 + bi * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
#pragma unroll
      for (int bj = 0; bj < 2; ++bj) {
        const int64_t gj = col0 + wn * 64 + bj * 32 + l32;
        if (gi >= r0 && gi < r1 && gj < n) out[(gi - r0) * n + gj] = acc[bi][bj][r];
      }
    }
}

// ------------------------------------------------------------------ launchers

hipError_t launch_gather_sorted(const float* Xp, const float* nrm, const IterBufs& b, const int* cl,
                                int64_t n_pad, int d_pad, float* Xs, float* nrm_s, int* cs,
                                hipStream_t s) {
  hipLaunchKernelGGL(gather_sorted_kernel, dim3((unsigned)((n_pad + 3) / 4)), dim3(256), 0, s, Xp,
                     nrm, b.perm, cl, b.n, n_pad, d_pad, b.k, Xs, nrm_s, cs);
  return hipGetLastError();
}

hipError_t launch_diag_from_norms(const float* nrm, int64_t n, const KappaParams& kp, float* diagK,
                                  hipStream_t s) {
  dim3 grid((unsigned)((n + 255) / 256));
  if (kp.kind == LINEAR) hipLaunchKernelGGL(diag_from_norms_kernel<LINEAR>, grid, dim3(256), 0, s, nrm, n, kp, diagK);
  else if (kp.kind == POLY) hipLaunchKernelGGL(diag_from_norms_kernel<POLY>, grid, dim3(256), 0, s, nrm, n, kp, diagK);
  else hipLaunchKernelGGL(diag_from_norms_kernel<GAUSS>, grid, dim3(256), 0, s, nrm, n, kp, diagK);
  return hipGetLastError();
}

int onthefly_segments(int64_t n) {
  const int nt = (int)((n + kTile - 1) / kTile);
  int nseg = (4096 + nt - 1) / nt;  // at least ~4096 workgroups: 8 per CU slot pair
  if (nseg > nt) nseg = nt;
  if (nseg > 64) nseg = 64;
  return nseg < 1 ? 1 : nseg;
}

hipError_t launch_onthefly(const float* Xs, const float* nrm_s, const int* cs,
                           const unsigned* maxnrm_bits, const IterBufs& b, int d_pad,
                           const KappaParams& kp, float* Epart, hipStream_t s) {
  const int nt = (int)((b.n + kTile - 1) / kTile), nseg = onthefly_segments(b.n);
  dim3 grid((unsigned)((int64_t)nt * nseg)), block(256);
  if (kp.kind == LINEAR)
    hipLaunchKernelGGL(onthefly_kernel<LINEAR>, grid, block, 0, s, Xs, nrm_s, cs, maxnrm_bits, b.n, d_pad, b.ld, nt, nseg, b.k, kp, Epart);
  else if (kp.kind == POLY)
    hipLaunchKernelGGL(onthefly_kernel<POLY>, grid, block, 0, s, Xs, nrm_s, cs, maxnrm_bits, b.n, d_pad, b.ld, nt, nseg, b.k, kp, Epart);
  else
    hipLaunchKernelGGL(onthefly_kernel<GAUSS>, grid, block, 0, s, Xs, nrm_s, cs, maxnrm_bits, b.n, d_pad, b.ld, nt, nseg, b.k, kp, Epart);
  return hipGetLastError();
}

hipError_t launch_onthefly_reduce(const IterBufs& b, const float* Epart, const int* cs, hipStream_t s) {
  const int nt = (int)((b.n + kTile - 1) / kTile), nseg = onthefly_segments(b.n);
  hipLaunchKernelGGL(onthefly_reduce_kernel, dim3((unsigned)(b.nstripes * b.k)), dim3(256), 0, s, b,
                     Epart, cs, nt, nseg);
  return hipGetLastError();
}

hipError_t launch_kernel_rows(const float* Xp, const float* nrm, const unsigned* maxnrm_bits,
                              int64_t n, int d_pad, const KappaParams& kp, int64_t r0, int64_t r1,
                              float* out, hipStream_t s) {
  const int nt = (int)((n + kTile - 1) / kTile);
  const int64_t R0 = r0 / kTile * kTile;
  const int64_t rt = (r1 - R0 + kTile - 1) / kTile;
  dim3 grid((unsigned)(rt * nt)), block(256);
  if (kp.kind == LINEAR)
    hipLaunchKernelGGL(kernel_rows_kernel<LINEAR>, grid, block, 0, s, Xp, nrm, maxnrm_bits, n, d_pad, R0, r0, r1, nt, kp, out);
  else if (kp.kind == POLY)
    hipLaunchKernelGGL(kernel_rows_kernel<POLY>, grid, block, 0, s, Xp, nrm, maxnrm_bits, n, d_pad, R0, r0, r1, nt, kp, out);
  else
    hipLaunchKernelGGL(kernel_rows_kernel<GAUSS>, grid, block, 0, s, Xp, nrm, maxnrm_bits, n, d_pad, R0, r0, r1, nt, kp, out);
  return hipGetLastError();
}

}  // namespace kkm
