// On-the-fly updates: K is never stored.  Every update recomputes the tiles
// of K = kappa(X X^T) on the fp32 matrix cores and folds them straight into
// E = K V^T, the paper's single-GPU sliding-window baseline (Section VI-D)
// done at tile granularity, with V one-hot instead of dense.
//
// The points are first gathered into cluster-sorted order (the same stable
// sort the resident path uses), so along a row of K the columns of one
// cluster form one contiguous run, and a block of 128 sorted rows spans few
// clusters.  K is symmetric, so only tiles (I, J) with I <= J are computed:
//   * row side: a workgroup owns row block I and sweeps a segment of column
//     tiles J >= I in order.  Each lane keeps, for each of its 32 rows, the
//     running sum of its own columns' entries; when the sweep leaves a cluster
//     the lanes' sums are reduced across the workgroup in a fixed order and
//     written as that cluster's partial for the segment.
//   * column side (J > I): the tile's column sums over the rows of I, one per
//     cluster run of those rows, are the row sums of block J over columns I
//     (K(i,j) = K(j,i)); they are written as partials of block J.
// A second kernel adds, for every sorted row and cluster, the row-side
// segment partials and the column-side partials of the earlier blocks, in a
// fixed order.  E comes out in sorted row order; the assign kernel reads it
// through the inverse permutation.
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

// Whether any Gaussian entry may need the fix-up, from the largest norm.
__device__ inline bool any_fix(const unsigned* maxnrm_bits, const KappaParams& kp) {
  const float m = __uint_as_float(*maxnrm_bits);
  return kp.kind == GAUSS && gauss_needs_fix(1.f, m, m, kp);
}

// One 128 x 128 tile of K from its B tile (acc), rows at row0 and columns at
// col0 of the staged points Y (n_pad x d_pad, column norms ny; rn[0..127]
// for the tile's rows: their norms, for the Gaussian scaled by
// c = -gamma log2(e) as gauss_scaled takes them): kappa applied, the Gaussian diagonal set to
// exactly 1, entries outside n x n zeroed, and (FIX) Gaussian entries flagged
// as cancellation-prone recomputed from the differences after the unrolled
// pass.  Row indices are block-local 32-bit values, so no per-row 64-bit
// index stays live across tiles.
template <int KIND, bool FIX>
__device__ inline void kappa_tile(floatx16 acc[2][2], const float* __restrict__ Y,
                                  const float* __restrict__ ny, const float* rn, int64_t n,
                                  int d_pad, int64_t row0, int64_t col0, const KappaParams& kp) {
  // u = c|x_i|^2 + c|x_j|^2 rounds the same for (i, j) and (j, i) only if
  // the products are not fused into the sum
#pragma clang fp contract(off)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1, l32 = lane & 31, h = lane >> 5;
  const int nrows = (int)(n - row0 < kTile ? n - row0 : kTile);
  const int ncols = (int)(n - col0 < kTile ? n - col0 : kTile);
  const bool diag = row0 == col0;
  const bool interior = nrows == kTile && ncols == kTile && !diag;
  const int rbase = wm * 64 + 4 * h, cbase = wn * 64 + l32;
  float cnj[2] = {0.f, 0.f};
  if (KIND == GAUSS) {
    cnj[0] = kp.neg_g_log2e * ny[col0 + cbase];
    cnj[1] = kp.neg_g_log2e * ny[col0 + cbase + 32];
  }
  bool flagged = false;  // some entry of this lane may need the fix-up
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int il = rbase + bi * 32 + 8 * (r >> 2) + (r & 3);
      const float cni = (KIND == GAUSS) ? rn[il] : 0.f;
#pragma unroll
      for (int bj = 0; bj < 2; ++bj) {
        const int jl = cbase + bj * 32;
        float v;
        if (KIND == GAUSS) {
          const float u = cni + cnj[bj];
          v = gauss_scaled(acc[bi][bj][r], u, kp);
          if (FIX) flagged |= gauss_needs_fix_scaled(v, u, kp);
        } else {
          v = kappa<KIND>(acc[bi][bj][r], 0.f, 0.f, kp);
        }
        if (!interior) {
          if (KIND == GAUSS && diag && il == jl) v = 1.f;
          if (il >= nrows || jl >= ncols) v = 0.f;
        }
        acc[bi][bj][r] = v;
      }
    }
  // Only where some lane of the wave flagged an entry is the exact set
  // formed: the entries off the diagonal whose estimate (on the value kept,
  // which outside n x n is 0) calls for the recomputation.
  if (KIND == GAUSS && FIX && __ballot(flagged)) {
    // the row norms are read again here rather than kept in registers
    // across the common path
    asm volatile("" ::: "memory");
    int rb = rbase, cb = cbase;
    asm volatile("" : "+v"(rb), "+v"(cb));
    unsigned long long fixmask = 0;
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int il = rb + bi * 32 + 8 * (r >> 2) + (r & 3);
        const float cni = rn[il];
#pragma unroll
        for (int bj = 0; bj < 2; ++bj) {
          const int jl = cb + bj * 32;
          if (gauss_needs_fix_scaled(acc[bi][bj][r], cni + cnj[bj], kp) && !(diag && il == jl))
            fixmask |= 1ull << ((bi * 2 + bj) * 16 + r);
        }
      }
    while (fixmask) {
      const int e = __ffsll((long long)fixmask) - 1;
      fixmask &= fixmask - 1;
      const int bi = e >> 5, bj = (e >> 4) & 1, r = e & 15;
      const int il = rb + bi * 32 + 8 * (r >> 2) + (r & 3), jl = cb + bj * 32;
      if (il < nrows && jl < ncols) {
        const float w = gauss_direct(Y + (row0 + il) * d_pad, Y + (col0 + jl) * d_pad, d_pad, kp);
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int p = 0; p < 2; ++p)
#pragma unroll
            for (int rr = 0; rr < 16; ++rr)
              if (q == bi && p == bj && rr == r) acc[q][p][rr] = w;
      }
    }
  }
}

// Segment bounds: segment s of nseg covers column tiles [seg_begin(s), seg_begin(s+1)).
__device__ __host__ inline int seg_begin(int s, int nt, int nseg) { return (int)((int64_t)s * nt / nseg); }

// bmax[P] = the largest squared norm among the sorted points of block P (128
// threads per block; padding rows hold 0): an upper bound of |x_i|^2 + |x_j|^2
// over a tile, with which the sweep skips the Gaussian fix-up estimate.
__global__ __launch_bounds__(128) void blockmax_kernel(const float* __restrict__ nrm_s, float* __restrict__ bmax) {
  __shared__ float part[2];
  float v = nrm_s[(int64_t)blockIdx.x * kTile + threadIdx.x];
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) bmax[blockIdx.x] = fmaxf(part[0], part[1]);
}

// Per update: for each row block P of the sorted order, the first cluster its
// rows hold (cA), how many clusters they span (nruns), and where its
// column-side partials start (cbase, in rows of 128 floats):
//   cbase[P] = sum_{P' < P} (nt - 1 - P') * nruns[P'].
// One workgroup: a thread per contiguous range of blocks, then a scan.
__global__ __launch_bounds__(1024) void onthefly_tables_kernel(const int* __restrict__ cs, int64_t n,
                                                               int nt, int* __restrict__ cA,
                                                               int* __restrict__ nruns,
                                                               int64_t* __restrict__ cbase) {
  __shared__ int64_t part[1024];
  const int tid = threadIdx.x;
  const int per = (nt + 1023) / 1024, lo = tid * per, hi = min(nt, lo + per);
  int64_t s = 0;
  for (int P = lo; P < hi; ++P) {
    const int64_t last = min((int64_t)P * kTile + kTile - 1, n - 1);
    const int a = cs[(int64_t)P * kTile], b = cs[last];
    cA[P] = a;
    nruns[P] = b - a + 1;
    s += (int64_t)(nt - 1 - P) * (b - a + 1);
  }
  part[tid] = s;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {  // inclusive scan (Hillis-Steele)
    const int64_t v = tid >= off ? part[tid - off] : 0;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  int64_t run = tid > 0 ? part[tid - 1] : 0;
  for (int P = lo; P < hi; ++P) {
    cbase[P] = run;
    run += (int64_t)(nt - 1 - P) * nruns[P];
  }
}

// FIX: the variant with the Gaussian fix-up path.  Both variants are
// launched; each returns at once unless the largest norm calls for it.
template <int KIND, bool FIX>
__global__ __launch_bounds__(256, 2) void onthefly_kernel(
    const float* __restrict__ Xs, const float* __restrict__ nrm_s, const int* __restrict__ cs,
    const unsigned* __restrict__ maxnrm_bits, const int* __restrict__ off,
    const int* __restrict__ cA, const int* __restrict__ nruns, const int64_t* __restrict__ cbase,
    int64_t n, int d_pad, int64_t ld, int nt, int nseg, int k, KappaParams kp,
    float* __restrict__ Epart, float* __restrict__ Cpart) {
  // The block's row norms sit after the mainloop buffers in the same array,
  // so the compiler reloads them per tile instead of pinning 32 registers.
  __shared__ __attribute__((aligned(16))) float lds[kLdsFloats + kTile];
  // Work items (segment s, row block I < seg_begin(s+1)), segment-major: the
  // hardware deals consecutive workgroups round-robin to the 8 XCDs, so every
  // XCD gets an even share, and the concurrent workgroups of one XCD sweep
  // the same column tiles (shared in its L2).
  int s = 0;
  int64_t first = 0;  // items before segment s
  while (s + 1 < nseg && first + seg_begin(s + 1, nt, nseg) <= (int64_t)blockIdx.x) {
    first += seg_begin(s + 1, nt, nseg);
    ++s;
  }
  const int I = (int)((int64_t)blockIdx.x - first);
  const int sb = seg_begin(s, nt, nseg), se = seg_begin(s + 1, nt, nseg);
  if (I >= se) return;  // only past the last item
  if (KIND == GAUSS && any_fix(maxnrm_bits, kp) != FIX) return;
  const int jt0 = sb > I ? sb : I, jt1 = se;
  const int64_t row0 = (int64_t)I * kTile;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, l32 = lane & 31, h = lane >> 5;
  const int runA = cA[I], nr = nruns[I];
  float* const cp = Cpart + cbase[I] * kTile;  // this block's column-side partials
  float* const rn = lds + kLdsFloats;
  if (tid < kTile) rn[tid] = (KIND == GAUSS ? kp.neg_g_log2e : 1.f) * nrm_s[row0 + tid];

  float rowacc[2][16];
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int r = 0; r < 16; ++r) rowacc[bi][r] = 0.f;

  // Row side: reduce the lanes' running sums over the columns of each row and
  // write them as cluster c's partial for this segment; fixed order.
  auto flush = [&](int c) {
    float* red = lds;  // [wm][wn][64], free between tiles
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
        if (l32 == 0) red[(wm * 2 + wn) * 64 + bi * 32 + 8 * (r >> 2) + 4 * h + (r & 3)] = v;
        rowacc[bi][r] = 0.f;
      }
    __syncthreads();
    if (wn == 0) {
      const int64_t gi = row0 + wm * 64 + lane;
      if (gi < n)
        Epart[((int64_t)s * k + c) * ld + gi] = red[(wm * 2) * 64 + lane] + red[(wm * 2 + 1) * 64 + lane];
    }
    __syncthreads();
  };

  // Column side of tile (I, J), J > I: column sums over the rows in sorted
  // positions [lo, hi) (all rows when the block holds one cluster) written as
  // run u of the tile's partials; fixed order.
  auto column_side = [&](int J, int u, bool all_rows, int lo, int hi, floatx16 (&a)[2][2]) {
    float c0 = 0.f, c1 = 0.f;
    const int llo = lo - (int)row0, lhi = hi - (int)row0;  // block-local row range
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        bool in = all_rows;
        if (!all_rows) {
          const int il = wm * 64 + bi * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
          in = il >= llo && il < lhi;
        }
        c0 += in ? a[bi][0][r] : 0.f;
        c1 += in ? a[bi][1][r] : 0.f;
      }
    c0 += __shfl_xor(c0, 32, 64);
    c1 += __shfl_xor(c1, 32, 64);
    float* csum = lds;  // [wm][128]
    if (h == 0) {
      csum[wm * 128 + wn * 64 + l32] = c0;
      csum[wm * 128 + wn * 64 + 32 + l32] = c1;
    }
    __syncthreads();
    if (tid < kTile) cp[((int64_t)(J - I - 1) * nr + u) * kTile + tid] = csum[tid] + csum[kTile + tid];
    __syncthreads();
  };

  int cur = cs[(int64_t)jt0 * kTile];
  floatx16 acc[2][2];
  for (int J = jt0; J < jt1; ++J) {
    const int64_t col0 = (int64_t)J * kTile;
    mma_tile(Xs + row0 * d_pad, Xs + col0 * d_pad, d_pad, lds, acc);
    kappa_tile<KIND, FIX>(acc, Xs, nrm_s, rn, n, d_pad, row0, col0, kp);
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
    if (J > I) {
      if (nr == 1) {
        column_side(J, 0, true, 0, 0, acc);
      } else {
        for (int u = 0; u < nr; ++u) column_side(J, u, false, off[runA + u], off[runA + u + 1], acc);
      }
    }
  }
  flush(cur);
}

// ---- Small widths (d_pad <= kRegMaxDpad): no barrier per tile.
//
// The block's 128 rows are staged in LDS once per work item; each wavefront
// (wm, wn) holds its 64 columns of the current tile J as MFMA operands in
// registers, loaded straight from the sorted points: lane (l, h) keeps
// column l of each 32-column block at k = h*HP .. h*HP + HP - 1 (HP =
// d_pad / 2), reads its rows at the same k from LDS, and step s of
// v_mfma_f32_32x32x2_f32 pairs k = s with k = HP + s.  The next tile's columns
// are loaded as soon as the current tile's products are issued, so the loads
// run beside the kappa epilogue.  The row side and the column side are kept
// per wavefront (two halves per partial: the wn halves of the row-side
// partials, the wm halves of the column-side partials), so the four
// wavefronts never wait for each other inside the sweep; two workgroups per
// CU give every SIMD two independent wavefronts, one streaming products while
// the other runs its epilogue.
// kappa on the wavefront's 64 x 64 block of an interior tile (off the
// diagonal, all rows and columns below n), as kappa_tile, laid out for the
// sweep's instruction budget: the Gaussian on norms scaled once and the
// fix-up estimate kept as one running minimum of u v per lane, so the
// per-entry test (and its mask) is formed only where some lane's minimum
// calls for it.  Diagonal and last tiles take kappa_tile.
template <int KIND, bool FIX>
__device__ inline void kappa_tile_interior(floatx16 (&acc)[2][2], const float* __restrict__ Y,
                                           const float* __restrict__ ny, const float* rn, int d_pad,
                                           int64_t row0, int64_t col0, const KappaParams& kp, bool tile_fix) {
  // u = c|x_i|^2 + c|x_j|^2 rounds the same for (i, j) and (j, i) only if
  // the products are not fused into the sum
#pragma clang fp contract(off)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1, l32 = lane & 31, h = lane >> 5;
  const int rbase = wm * 64 + 4 * h, cbase = wn * 64 + l32;
  float cnj[2] = {0.f, 0.f};
  if (KIND == GAUSS) {
    cnj[0] = kp.neg_g_log2e * ny[col0 + cbase];
    cnj[1] = kp.neg_g_log2e * ny[col0 + cbase + 32];
  }
  float umin = 0.f;  // min over this lane's entries of u v (the fix-up estimate)
  auto pass = [&](bool est) {
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float4 r4 = {0.f, 0.f, 0.f, 0.f};
        if (KIND == GAUSS) r4 = *(const float4*)(rn + rbase + bi * 32 + 8 * q);
        const float cn[4] = {r4.x, r4.y, r4.z, r4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int bj = 0; bj < 2; ++bj) {
            const float a = acc[bi][bj][4 * q + e];
            if (KIND == GAUSS) {
              const float u = cn[e] + cnj[bj];
              const float v = gauss_scaled(a, u, kp);
              if (est) umin = fminf(umin, u * v);
              acc[bi][bj][4 * q + e] = v;
            } else {
              acc[bi][bj][4 * q + e] = kappa<KIND>(a, 0.f, 0.f, kp);
            }
          }
      }
  };
  // the estimate only where the tile's largest norms allow an entry to need
  // the fix-up (uniform); elsewhere the plain pass
  if (KIND == GAUSS && FIX && tile_fix) pass(true);
  else pass(false);
  if (KIND == GAUSS && FIX && tile_fix && __ballot(umin < kp.fix_uthr)) {
    // the lane's row base is made opaque, so the per-entry index work is
    // formed here and not hoisted out of the sweep
    asm volatile("" ::: "memory");
    int rb = rbase;
    asm volatile("" : "+v"(rb));
    unsigned long long fixmask = 0;
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float cni = rn[rb + bi * 32 + 8 * (r >> 2) + (r & 3)];
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
          if (gauss_needs_fix_scaled(acc[bi][bj][r], cni + cnj[bj], kp)) fixmask |= 1ull << ((bi * 2 + bj) * 16 + r);
      }
    while (fixmask) {
      const int e = __ffsll((long long)fixmask) - 1;
      fixmask &= fixmask - 1;
      const int bi = e >> 5, bj = (e >> 4) & 1, r = e & 15;
      const int il = rb + bi * 32 + 8 * (r >> 2) + (r & 3), jl = cbase + bj * 32;
      const float w = gauss_direct(Y + (row0 + il) * d_pad, Y + (col0 + jl) * d_pad, d_pad, kp);
#pragma unroll
      for (int qq = 0; qq < 2; ++qq)
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
          for (int rr = 0; rr < 16; ++rr)
            if (qq == bi && p == bj && rr == r) acc[qq][p][rr] = w;
    }
  }
}

template <int KIND, bool FIX, int HP>
__global__ __launch_bounds__(256, 2) void onthefly_reg_kernel(
    const float* __restrict__ Xs, const float* __restrict__ nrm_s, const int* __restrict__ cs,
    const unsigned* __restrict__ maxnrm_bits, const int* __restrict__ off,
    const int* __restrict__ cA, const int* __restrict__ nruns, const int64_t* __restrict__ cbase,
    const float* __restrict__ bmax, int64_t n, int64_t ld, int nt, int nseg, int k, KappaParams kp,
    float* __restrict__ Epart, float* __restrict__ Cpart) {
  constexpr int d_pad = 2 * HP, ldsA = 2 * HP + 4;
  __shared__ __attribute__((aligned(16))) float rn[kTile];
  __shared__ __attribute__((aligned(16))) float As[kTile * ldsA];
  // work items as in onthefly_kernel: (segment s, row block I), segment-major
  int s = 0;
  int64_t first = 0;
  while (s + 1 < nseg && first + seg_begin(s + 1, nt, nseg) <= (int64_t)blockIdx.x) {
    first += seg_begin(s + 1, nt, nseg);
    ++s;
  }
  const int I = (int)((int64_t)blockIdx.x - first);
  const int sb = seg_begin(s, nt, nseg), se = seg_begin(s + 1, nt, nseg);
  if (I >= se) return;
  if (KIND == GAUSS && any_fix(maxnrm_bits, kp) != FIX) return;
  const int jt0 = sb > I ? sb : I, jt1 = se;
  const int64_t row0 = (int64_t)I * kTile;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, l32 = lane & 31, h = lane >> 5;
  const int runA = cA[I], nr = nruns[I];
  // this block's column-side partials: rows of 2 x 128 floats (the wm halves)
  float* const cp = Cpart + cbase[I] * (2 * kTile);
  if (tid < kTile) rn[tid] = (KIND == GAUSS ? kp.neg_g_log2e : 1.f) * nrm_s[row0 + tid];

  for (int f = tid; f < kTile * (HP / 2); f += 256) {  // the block's rows, 16 bytes per thread and step
    const int r = f / (HP / 2), c = f % (HP / 2);
    *(float4*)(As + r * ldsA + 4 * c) = *(const float4*)(Xs + (row0 + r) * d_pad + 4 * c);
  }
  __syncthreads();  // rn, As
  const float* const Aw = As + wm * 64 * ldsA;

  float rowacc[2][16];
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int r = 0; r < 16; ++r) rowacc[bi][r] = 0.f;

  // Row side: this wavefront's running sums over its 64 columns, reduced over
  // the lanes (fixed xor tree) and written as cluster c's partial of segment
  // s, half wn.
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
        rowacc[bi][r] = v;
      }
    if (l32 == 0) {
      float* ep = Epart + (((int64_t)s * k + c) * 2 + wn) * ld + row0;
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int il = wm * 64 + bi * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
          if (row0 + il < n) ep[il] = rowacc[bi][r];
        }
    }
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 16; ++r) rowacc[bi][r] = 0.f;
  };

  // Column side of tile (I, J), J > I, for this wavefront's 64 rows and 64
  // columns: the column sums over the rows in sorted positions [lo, hi) (all
  // rows when the block holds one cluster), written as run u, half wm.
  auto column_side = [&](int J, int u, bool all_rows, int lo, int hi, const floatx16 (&t)[2][2]) {
    float c0 = 0.f, c1 = 0.f;
    const int llo = lo - (int)row0, lhi = hi - (int)row0;
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        bool in = all_rows;
        if (!all_rows) {
          const int il = wm * 64 + bi * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
          in = il >= llo && il < lhi;
        }
        c0 += in ? t[bi][0][r] : 0.f;
        c1 += in ? t[bi][1][r] : 0.f;
      }
    c0 += __shfl_xor(c0, 32, 64);
    c1 += __shfl_xor(c1, 32, 64);
    if (h == 0) {
      float* dst = cp + ((int64_t)(J - I - 1) * nr + u) * (2 * kTile) + wm * kTile + wn * 64 + l32;
      dst[0] = c0;
      dst[32] = c1;
    }
  };

  // The clusters are walked over the whole tile's columns (not only this
  // wavefront's half), so both halves write a partial, possibly zero, for
  // every cluster the segment's columns hold.
  int cur = cs[(int64_t)jt0 * kTile];
  floatx16 acc[2][2];
  for (int J = jt0; J < jt1; ++J) {
    const int64_t col0 = (int64_t)J * kTile;
    {
      float b[2][HP];
#pragma unroll
      for (int q = 0; q < 2; ++q) load_operand<HP>(Xs, col0 + wn * 64 + q * 32 + l32, d_pad, h, b[q]);
      mma_rows_lds<HP>(Aw, b[0], acc[0][0], acc[1][0], l32, h);
      mma_rows_lds<HP>(Aw, b[1], acc[0][1], acc[1][1], l32, h);
    }
    // the epilogue's loads (row norms, column norms and ids) are not hoisted
    // into the product loop, where they would hold registers
    __builtin_amdgcn_sched_barrier(0);
    if (J == I || col0 + kTile > n)  // uniform: the diagonal tile, the last tile
      kappa_tile<KIND, FIX>(acc, Xs, nrm_s, rn, n, d_pad, row0, col0, kp);
    else
      kappa_tile_interior<KIND, FIX>(acc, Xs, nrm_s, rn, d_pad, row0, col0, kp,
                                     FIX && gauss_needs_fix(1.f, bmax[I], bmax[J], kp));
    {
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
    if (J > I) {
      if (nr == 1) {
        column_side(J, 0, true, 0, 0, acc);
      } else {
        for (int u = 0; u < nr; ++u) column_side(J, u, false, off[runA + u], off[runA + u + 1], acc);
      }
    }
  }
  flush(cur);
}

int onthefly_halves(int d_pad) { return d_pad <= kRegMaxDpad ? 2 : 1; }

hipError_t launch_blockmax(const float* nrm, int64_t nblocks, float* bmax, hipStream_t s) {
  hipLaunchKernelGGL(blockmax_kernel, dim3((unsigned)nblocks), dim3(kTile), 0, s, nrm, bmax);
  return hipGetLastError();
}

// Workgroup (stripe, j): E^T_sorted(j, q) for the stripe's sorted rows q:
//   the row-side partials of the segments that block Q = q/128 swept over
//   columns of cluster j, in segment order, then the column-side partials of
//   the blocks P < Q holding rows of cluster j, in block order;
// plus the stripe's part of sum_{q in L_j} E(q, j) in fp64 (cs[q] == j).
// halves: 2 when the sweep kept per-wavefront partials (two per row-side
// partial and two per column-side partial, added in order), else 1.
__global__ __launch_bounds__(256) void onthefly_reduce_kernel(
    IterBufs b, const float* __restrict__ Epart, const float* __restrict__ Cpart,
    const int* __restrict__ cs, const int* __restrict__ cA, const int* __restrict__ nruns,
    const int64_t* __restrict__ cbase, int nt, int nseg, int halves) {
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
    const int Q = (int)(col / kTile);
    f4 e = {0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < nseg; ++s) {
      const int sb = seg_begin(s, nt, nseg), se = seg_begin(s + 1, nt, nseg);
      if (se <= Q) continue;
      const int64_t c0 = (int64_t)(sb > Q ? sb : Q) * kTile;
      const int64_t c1 = (int64_t)se * kTile < b.n ? (int64_t)se * kTile : b.n;
      if (c0 < hi && lo < c1)
        for (int hh = 0; hh < halves; ++hh)
          e += *(const f4*)(Epart + (((int64_t)s * b.k + j) * halves + hh) * ld + col);
    }
    const int Pl = (hi - 1) / kTile;
    for (int P = lo / kTile; P <= Pl && P < Q; ++P) {
      const float* cr = Cpart + (cbase[P] + (int64_t)(Q - P - 1) * nruns[P] + (j - cA[P])) * (halves * kTile) +
                        (col - (int64_t)Q * kTile);
      for (int hh = 0; hh < halves; ++hh) e += *(const f4*)(cr + hh * kTile);
    }
    *(f4*)(b.Et + (int64_t)j * ld + col) = e;
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (col + c < b.n && cs[col + c] == j) zs += (double)e[c];
  }
  for (int o = 32; o > 0; o >>= 1) zs += __shfl_xor(zs, o, 64);
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
  __shared__ __attribute__((aligned(16))) float lds[kLdsFloats + kTile];
  const int J = (int)(blockIdx.x % (unsigned)nt), I = (int)(blockIdx.x / (unsigned)nt);
  const int64_t row0 = R0 + (int64_t)I * kTile, col0 = (int64_t)J * kTile;
  float* const rn = lds + kLdsFloats;
  if (threadIdx.x < kTile) rn[threadIdx.x] = (KIND == GAUSS ? kp.neg_g_log2e : 1.f) * nrm[row0 + threadIdx.x];
  floatx16 acc[2][2];
  mma_tile(Xp + row0 * d_pad, Xp + col0 * d_pad, d_pad, lds, acc);
  if (any_fix(maxnrm_bits, kp)) kappa_tile<KIND, true>(acc, Xp, nrm, rn, n, d_pad, row0, col0, kp);
  else kappa_tile<KIND, false>(acc, Xp, nrm, rn, n, d_pad, row0, col0, kp);
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
  int nseg = (8192 + nt - 1) / nt;  // ~4096 workgroups right of the diagonal
  if (nseg > nt) nseg = nt;
  if (nseg > 64) nseg = 64;
  return nseg < 1 ? 1 : nseg;
}

int64_t onthefly_cpart_floats(int64_t n, int k) {
  const int64_t nt = (n + kTile - 1) / kTile;
  // sum_P (nt-1-P) * nruns[P] with sum_P nruns[P] <= nt + k - 1
  return (nt * (nt - 1) / 2 + (int64_t)(k - 1) * (nt > 0 ? nt - 1 : 0)) * kTile + kTile;
}

hipError_t launch_onthefly(const float* Xs, const float* nrm_s, const int* cs,
                           const unsigned* maxnrm_bits, const IterBufs& b, int d_pad,
                           const KappaParams& kp, const OtfTables& tb, float* Epart, float* Cpart,
                           hipStream_t s) {
  const int nt = (int)((b.n + kTile - 1) / kTile), nseg = onthefly_segments(b.n);
  hipLaunchKernelGGL(onthefly_tables_kernel, dim3(1), dim3(1024), 0, s, cs, b.n, nt, tb.cA,
                     tb.nruns, tb.cbase);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  int64_t items = 0;  // (segment, row block) pairs right of the diagonal
  for (int q = 0; q < nseg; ++q) items += seg_begin(q + 1, nt, nseg);
  dim3 grid((unsigned)items), block(256);
  if (d_pad <= kRegMaxDpad) {
    if (d_pad % 8) return hipErrorInvalidValue;
    if (kp.kind == GAUSS) {
      hipLaunchKernelGGL(blockmax_kernel, dim3((unsigned)nt), dim3(kTile), 0, s, nrm_s, tb.bmax);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
#define KKM_OTF_REG(KIND, FIX, HP)                                                                          \
  hipLaunchKernelGGL((onthefly_reg_kernel<KIND, FIX, HP>), grid, block, 0, s, Xs, nrm_s, cs, maxnrm_bits, b.off, \
                     tb.cA, tb.nruns, tb.cbase, tb.bmax, b.n, b.ld, nt, nseg, b.k, kp, Epart, Cpart)
#define KKM_OTF_REG_HP(KIND, FIX)           \
  switch (d_pad / 2) {                      \
    case 4: KKM_OTF_REG(KIND, FIX, 4); break;   \
    case 8: KKM_OTF_REG(KIND, FIX, 8); break;   \
    case 12: KKM_OTF_REG(KIND, FIX, 12); break; \
    case 16: KKM_OTF_REG(KIND, FIX, 16); break; \
    case 20: KKM_OTF_REG(KIND, FIX, 20); break; \
    case 24: KKM_OTF_REG(KIND, FIX, 24); break; \
    case 28: KKM_OTF_REG(KIND, FIX, 28); break; \
    default: KKM_OTF_REG(KIND, FIX, 32); break; \
  }
    if (kp.kind == LINEAR) {
      KKM_OTF_REG_HP(LINEAR, false);
    } else if (kp.kind == POLY) {
      KKM_OTF_REG_HP(POLY, false);
    } else {
      KKM_OTF_REG_HP(GAUSS, false);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
      KKM_OTF_REG_HP(GAUSS, true);
    }
#undef KKM_OTF_REG_HP
#undef KKM_OTF_REG
    return hipGetLastError();
  }
  if (kp.kind == LINEAR) {
    hipLaunchKernelGGL((onthefly_kernel<LINEAR, false>), grid, block, 0, s, Xs, nrm_s, cs, maxnrm_bits,
                       b.off, tb.cA, tb.nruns, tb.cbase, b.n, d_pad, b.ld, nt, nseg, b.k, kp, Epart, Cpart);
  } else if (kp.kind == POLY) {
    hipLaunchKernelGGL((onthefly_kernel<POLY, false>), grid, block, 0, s, Xs, nrm_s, cs, maxnrm_bits,
                       b.off, tb.cA, tb.nruns, tb.cbase, b.n, d_pad, b.ld, nt, nseg, b.k, kp, Epart, Cpart);
  } else {
    hipLaunchKernelGGL((onthefly_kernel<GAUSS, false>), grid, block, 0, s, Xs, nrm_s, cs, maxnrm_bits,
                       b.off, tb.cA, tb.nruns, tb.cbase, b.n, d_pad, b.ld, nt, nseg, b.k, kp, Epart, Cpart);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((onthefly_kernel<GAUSS, true>), grid, block, 0, s, Xs, nrm_s, cs, maxnrm_bits,
                       b.off, tb.cA, tb.nruns, tb.cbase, b.n, d_pad, b.ld, nt, nseg, b.k, kp, Epart, Cpart);
  }
  return hipGetLastError();
}

hipError_t launch_onthefly_reduce(const IterBufs& b, const float* Epart, const float* Cpart,
                                  const int* cs, const OtfTables& tb, int d_pad, hipStream_t s) {
  const int nt = (int)((b.n + kTile - 1) / kTile), nseg = onthefly_segments(b.n);
  hipLaunchKernelGGL(onthefly_reduce_kernel, dim3((unsigned)(b.nstripes * b.k)), dim3(256), 0, s, b,
                     Epart, Cpart, cs, tb.cA, tb.nruns, tb.cbase, nt, nseg, onthefly_halves(d_pad));
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
