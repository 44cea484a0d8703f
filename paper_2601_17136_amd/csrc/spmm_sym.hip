// One-hot SpMM over the packed (upper block triangle) K.
//
// E^T = V K (Eq. 4 in the E^T form of Section IV) with K symmetric and only
// tiles I <= J stored: a stored entry K(r, c) belongs to both
//   row side     E^T(cl(r), c) += K(r, c)   (every stored entry), and
//   column side  E^T(cl(c), r) += K(r, c)   (entries right of r's diagonal tile),
// so each stored byte is read once and serves two sums.  The rows are taken
// in cluster-sorted chunks of at most 64 or 128 rows (all in one cluster), so
// the row side is a plain column sum over the chunk, as in the full-storage
// SpMM.  The column side needs, for every row, its entries summed per label
// of their column: a product with the one-hot matrix of the column labels,
// which runs on the fp32 matrix cores (v_mfma_f32_16x16x4_f32, 16 labels per
// block, exact: every product is 0 or the entry itself).
//
// Workgroup (chunk q, segment sg): NW wavefronts (4 or 8), one 16-row group
// each, over the column tiles of segment sg (BSEG tiles) that the chunk's
// rows store.
// Per tile a wavefront
//  - streams its 16 rows x 128 columns with 16-byte loads, two rows of 512
//    contiguous bytes per instruction, one tile ahead: a single register
//    buffer, refilled as soon as the block is staged (two buffers and two
//    tiles in flight measured slower: 180 vs 166 us on 20000 points);
//  - adds the rows in registers (row side), combines the wavefronts in LDS
//    and writes the chunk's partial P[q] for the tile;
//  - stages the block in LDS in two 64-column halves and reads each back in
//    the MFMA operand layout (lane = row, k slot = column) for the column
//    side.
// The scatter prepares, once per update, each sorted row's packed offset and
// each column tile's one-hot bits, so a workgroup's prologue is two parallel
// loads.  The column-side sums of a row stay in the accumulators for the whole
// segment and go to Ecp[sg] at sorted positions; ecol_sum_kernel adds the
// segments into Ecol at each row's point index, and spmm_reduce_sym_kernel
// adds them into E^T.  Fixed orders
// throughout, so the result is bitwise reproducible.
#include "kkm_internal.h"

#include <algorithm>
#include <climits>

namespace kkm {

typedef float f4 __attribute__((ext_vector_type(4)));

namespace {

// 90 VGPRs and ~23 KB (NW = 4) or ~45 KB (NW = 8) of LDS per workgroup:
// 20 or 16 wavefronts per CU.  Six wavefronts per SIMD (80 VGPRs, spilling)
// measured slower.
template <int NB, int NW, int BSEG>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(4))) void spmm_sym_kernel(
    const float* __restrict__ Kp, IterBufs b) {
  constexpr int R = 16 * NW, NT = 64 * NW;
  const int nseg = b.nseg;
  const int q = (int)(blockIdx.x / (unsigned)nseg), sg = (int)(blockIdx.x % (unsigned)nseg);
  // q < qmax, so the chunk table is read before the count says whether q is
  // in use (one round trip instead of two)
  const int nq = *b.nchunks, p0 = b.chunk_p0[q], p1 = b.chunk_p1[q], c0 = b.chunk_c0[q];
  const int Js = sg * BSEG, Je = min(b.nt, Js + BSEG);
  // Rows are in increasing index order within a chunk, so the first row has
  // the smallest tile; a segment left of it holds nothing of this chunk.
  if (q >= nq || c0 >= Je * kTile) return;
  const int nr = p1 - p0;

  __shared__ int rtile[R];
  __shared__ int64_t roff[R];
  __shared__ unsigned mskl[BSEG][NB][4][16];     // one-hot bits: [tile][label block][k slot][label]
  __shared__ f4 tile[NW][16 * 16];                // per wavefront: 16 rows x 16 chunks of 16 B (a half tile)
  __shared__ f4 red[2][NW][32];                   // row-side sums of the wavefronts

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int li = lane & 15, lk = lane >> 4;   // MFMA layout: row li, k slot lk
  const int h = lane >> 5, c32 = lane & 31;   // load layout: row 2g + h, columns 4*c32 .. +3
  const int64_t ld = b.ld, n = b.n;

  // Row tiles and packed row offsets, and the segment's one-hot bits (bit
  // 4g+e of [tile][nb][lk][li]: column 16g + 4lk + e of the tile has label
  // 16nb + li), all prepared by the scatter for this update.
  if (tid < R) {
    if (tid < nr) {
      rtile[tid] = b.perm[p0 + tid] / kTile;
      roff[tid] = b.roffp[p0 + tid];
    } else {
      rtile[tid] = INT_MAX;
      roff[tid] = 0;
    }
  }
  for (int t = tid; t < (Je - Js) * NB * 64; t += NT)
    (&mskl[0][0][0][0])[t] = b.mskg[(int64_t)Js * NB * 64 + t];
  __syncthreads();

  const int I0 = rtile[0];
  const int J_lo = max(Js, I0), J_hi = Je;
  const int um = w * 16 + li;  // this lane's row in the MFMA layout
  const int rt_m = rtile[um];
  const int rt_first = rtile[w * 16], rt_last = rtile[min(w * 16 + 15, nr - 1)];
  f4 D[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) D[nb] = f4{0.f, 0.f, 0.f, 0.f};
  f4 bb[8];
  f4* tw = tile[w];

  // Rows not stored in tile J (their diagonal tile is further right) and rows
  // past the chunk read the zero page instead.
  auto load = [&](f4(&buf)[8], int J) {
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      const int u = w * 16 + 2 * g + h;
      const bool on = rtile[u] <= J;
      const float* rp = on ? Kp + roff[u] + (int64_t)J * kTile + 4 * c32 : b.zero + 4 * c32;
      buf[g] = __builtin_nontemporal_load((const f4*)rp);
    }
  };

  auto step = [&](f4(&buf)[8], int J, int par) {
    // row side: this lane's 4 columns over its 8 rows, then the other half-wave's 8
    f4 rs = buf[0];
#pragma unroll
    for (int g = 1; g < 8; ++g) rs += buf[g];
#pragma unroll
    for (int e = 0; e < 4; ++e) rs[e] += __shfl_xor(rs[e], 32, 64);

    // column side: entries right of the row's own diagonal tile
    const int bi = J - Js;
    unsigned msk[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) msk[nb] = mskl[bi][nb][lk][li];
    const bool diag = rt_first <= J && J <= rt_last;  // some row of the group sits in tile J
    const bool dz = rt_m >= J;
    const bool any = rt_first < J || diag;
    // the block is staged and multiplied in two 64-column halves (chunk
    // index xor row keeps both access patterns conflict-free)
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      if ((c32 >> 4) == half) {
#pragma unroll
        for (int g = 0; g < 8; ++g) {
          const int r = 2 * g + h;
          tw[r * 16 + ((c32 & 15) ^ r)] = buf[g];
        }
      }
      if (half == 1) {
        // the whole block is staged: fetch the next tile into the buffer
        __builtin_amdgcn_sched_barrier(0);
        if (J + 1 < J_hi) load(buf, J + 1);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (any) {
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const int g = 4 * half + g4;
          f4 v = tw[li * 16 + ((4 * g4 + lk) ^ li)];  // row li, columns 16g + 4lk .. +3
          if (diag && dz) v = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int e = 0; e < 4; ++e)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
              const float a = (float)((msk[nb] >> (4 * g + e)) & 1u);
              D[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, v[e], D[nb], 0, 0, 0);
            }
        }
      }
    }

    // row side across the wavefronts -> P[q], columns of tile J
    if (h == 0) red[par][w][c32] = rs;
    __syncthreads();
    if (tid < kTile) {
      const float* rr = (const float*)red[par];
      float t = rr[tid];
#pragma unroll
      for (int ww = 1; ww < NW; ++ww) t += rr[ww * kTile + tid];
      b.P[(int64_t)q * ld + (int64_t)J * kTile + tid] = t;
    }
  };

  load(bb, J_lo);
  for (int J = J_lo; J < J_hi; ++J) step(bb, J, (J - J_lo) & 1);

  // D[nb][r]: label 16nb + 4lk + r of row um
  if (um < nr)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int lab = 16 * nb + 4 * lk + r;
        if (lab < b.k) b.Ecp[((int64_t)sg * b.k + lab) * n + p0 + um] = D[nb][r];
      }
}

// Ecol[j][perm[p]] = sum over the segments that hold the stored columns of
// the row at sorted position p, in order (stored at the point's own index, so
// the reduction reads it in step with E^T).  One output per thread: (chunk,
// label, row) over ecol_wgs(b) workgroups per chunk.
__device__ __host__ inline int ecol_wgs(const IterBufs& b) { return (b.k * b.chunk_len + 255) / 256; }
__global__ __launch_bounds__(256) void ecol_sum_kernel(IterBufs b) {
  const int per = ecol_wgs(b);
  const int q = (int)(blockIdx.x / (unsigned)per), part = (int)(blockIdx.x % (unsigned)per);
  const int nq = *b.nchunks, p0 = b.chunk_p0[q], p1 = b.chunk_p1[q], c0 = b.chunk_c0[q];
  if (q >= nq) return;
  const int nr = p1 - p0;
  const int t = part * 256 + (int)threadIdx.x;
  if (t >= b.k * nr) return;
  const int j = t / nr, u = t % nr;
  const int row = b.perm[p0 + u];
  const int s0 = c0 / kTile / b.bseg, last = b.nseg - 1;
  const int64_t seg_stride = (int64_t)b.k * b.n;
  const float* e = b.Ecp + (int64_t)j * b.n + p0 + u;
  float acc = 0.f;
  for (int sg = s0; sg <= last; sg += 8) {  // eight loads in flight, added in order
    float v[8];
#pragma unroll
    for (int x = 0; x < 8; ++x) v[x] = e[min(sg + x, last) * seg_stride];
#pragma unroll
    for (int x = 0; x < 8; ++x)
      if (sg + x <= last) acc += v[x];
  }
  b.Ecol[(int64_t)j * b.n + row] = acc;
}

// Workgroup (stripe of kSymRedStripe columns, cluster j).  Cluster j's many
// short chunks are split into four fixed quarters, one per wavefront, each
// summed in chunk order (a chunk's partial starts at its first stored
// column), and the quarters are added in order.  Then the column-side sums
// of the stripe's rows, and the stripe's part of sum_{i in L_j} E(i, j).
__global__ __launch_bounds__(256) void spmm_reduce_sym_kernel(IterBufs b, const int* __restrict__ cl) {
  const int ns = b.nzpart;
  const int stripe = (int)(blockIdx.x % (unsigned)ns), j = (int)(blockIdx.x / (unsigned)ns);
  const int qa = b.qfirst[j], qb = b.qfirst[j + 1];
  if (qa == qb) return;  // empty cluster: E^T(j, .) and z_j are never read
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  __shared__ f4 part[4][64];
  const int64_t ld = b.ld, n = b.n;
  const int64_t col = (int64_t)stripe * kSymRedStripe + 4 * lane;
  // the column-side sums and ids of the stripe's points, for wavefront 0's
  // epilogue, are loaded before the chunk loop
  float ec[4];
  int cc[4];
  if (w == 0) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int64_t x = min(col + c, n - 1);
      ec[c] = b.Ecol[(int64_t)j * n + x];
      cc[c] = cl[x];
    }
  }
  const int per = (qb - qa + 3) / 4;
  const int q0 = qa + w * per, q1 = min(qb, q0 + per);
  f4 e = {0.f, 0.f, 0.f, 0.f};
  if (col < ld) {
    // a chunk's partial starts at its first stored column; entries left of
    // it are stale and are read but not added
    for (int q = q0; q < q1; q += 8) {  // eight chunks in flight, added in order
      int c0[8];
      f4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int qq = min(q + u, q1 - 1);
        c0[u] = b.chunk_c0[qq];
        v[u] = *(const f4*)(b.P + (int64_t)qq * ld + col);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (q + u < q1 && col >= c0[u]) e += v[u];
    }
  }
  part[w][lane] = e;
  __syncthreads();
  if (w != 0) return;
  double zs = 0.0;
  if (col < ld) {
    e = (part[0][lane] + part[1][lane]) + (part[2][lane] + part[3][lane]);
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (col + c < n) e[c] += ec[c];
    *(f4*)(b.Et + (int64_t)j * ld + col) = e;
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (col + c < n && cc[c] == j) zs += (double)e[c];
  }
  for (int off = 32; off > 0; off >>= 1) zs += __shfl_xor(zs, off, 64);
  if (lane == 0) b.zpart[(int64_t)j * ns + stripe] = zs;
}

// Rows r0 .. r1-1 of the full K from the packed triangle.
__global__ __launch_bounds__(256) void packed_rows_kernel(const float* __restrict__ Kp, int64_t n,
                                                          int64_t ld, int64_t r0, int64_t r1,
                                                          float* __restrict__ out) {
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (c >= n) return;
  for (int64_t r = r0 + blockIdx.y; r < r1; r += gridDim.y) {
    const int64_t c0 = (r / kTile) * kTile;
    out[(r - r0) * n + c] = c >= c0 ? Kp[packed_row(r, ld) + c] : Kp[packed_row(c, ld) + r];
  }
}

}  // namespace

hipError_t launch_spmm_sym(const float* Kp, const IterBufs& b, hipStream_t s) {
  const unsigned grid = (unsigned)((int64_t)b.qmax * b.nseg);
  const int nb = b.nlb;
  if (nb != (b.k + 15) / 16) return hipErrorInvalidValue;
#define KKM_SYM_LAUNCH(NB, NW, S) \
  hipLaunchKernelGGL((spmm_sym_kernel<NB, NW, S>), dim3(grid), dim3(64 * NW), 0, s, Kp, b)
  if (b.chunk_len != 64 && b.chunk_len != 128) return hipErrorInvalidValue;
  if (b.bseg != 8 && !(b.bseg == 16 && nb == 1 && b.chunk_len == 128)) return hipErrorInvalidValue;
  const bool tall = b.chunk_len == 128;
  switch (nb) {
    case 1:
      if (b.bseg == 16) KKM_SYM_LAUNCH(1, 8, 16);
      else if (tall) KKM_SYM_LAUNCH(1, 8, 8);
      else KKM_SYM_LAUNCH(1, 4, 8);
      break;
    case 2: if (tall) KKM_SYM_LAUNCH(2, 8, 8); else KKM_SYM_LAUNCH(2, 4, 8); break;
    case 3: if (tall) KKM_SYM_LAUNCH(3, 8, 8); else KKM_SYM_LAUNCH(3, 4, 8); break;
    case 4: if (tall) KKM_SYM_LAUNCH(4, 8, 8); else KKM_SYM_LAUNCH(4, 4, 8); break;
    default: return hipErrorInvalidValue;  // k > kSymMaxK is rejected before launch
  }
#undef KKM_SYM_LAUNCH
  return hipGetLastError();
}

hipError_t launch_ecol_sum(const IterBufs& b, hipStream_t s) {
  hipLaunchKernelGGL(ecol_sum_kernel, dim3((unsigned)((int64_t)b.qmax * ecol_wgs(b))), dim3(256), 0, s, b);
  return hipGetLastError();
}

hipError_t launch_spmm_reduce_sym(const IterBufs& b, const int* cl, hipStream_t s) {
  hipLaunchKernelGGL(spmm_reduce_sym_kernel, dim3((unsigned)(b.nzpart * b.k)), dim3(256), 0, s, b, cl);
  return hipGetLastError();
}

hipError_t launch_packed_rows(const float* Kp, int64_t n, int64_t ld, int64_t r0, int64_t r1,
                              float* out, hipStream_t s) {
  const unsigned gy = (unsigned)std::min<int64_t>(r1 - r0, 65535);
  hipLaunchKernelGGL(packed_rows_kernel, dim3((unsigned)((n + 255) / 256), gy), dim3(256), 0, s, Kp,
                     n, ld, r0, r1, out);
  return hipGetLastError();
}

}  // namespace kkm
