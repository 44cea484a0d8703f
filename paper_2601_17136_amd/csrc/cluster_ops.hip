// The clustering iteration over a stored K (Section II-B, Eqs. 3-8; the loop
// body of Alg. 1 with a single process).
//
// E = K V^T is computed in its transposed form E^T = V K, the form the paper
// uses for its SpMM (Section IV): row j of E^T is the sum of the rows of K
// that belong to cluster j.  Points are first sorted by cluster (a stable
// counting sort), so every workgroup of the SpMM sums a run of rows of one
// cluster over a stripe of columns with a single accumulator: one add per
// element of K, each row segment read as 4 KB of contiguous memory.  K is
// symmetric, so the columns of E^T are the rows of E.
//
// Per update:  scatter (sorted order, chunk table)  ->  spmm_onehot (chunk
// partial sums)  ->  spmm_reduce (E^T, partial self-terms)  ->  assign (z,
// distances, argmin, new sizes, per-block histograms for the next scatter).
// All reductions of floating-point values run in a fixed order, so results
// are bitwise reproducible; only integer counters use atomics, and no kernel
// waits on another workgroup: every hand-off is a kernel boundary.
#include "kkm_internal.h"

#include <algorithm>

namespace kkm {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));

__device__ inline int clamp_id(int c, int k) { return c < 0 ? 0 : (c >= k ? k - 1 : c); }

// ----------------------------------------------------------------- assign
//
// mode 0 (labels): check ids, cluster sizes and per-block histograms.
// mode 1 (full):   z_j = (1/|L_j|^2) sum_s zpart[j][s]            (Eqs. 5-7)
//                  D(i,j) = K(i,i) - 2 E(i,j)/|L_j| + z_j         (Eq. 8 + diag K)
//                  cl'(i) = lowest j attaining min_j D(i,j); sizes of cl'.
// The per-block histograms (cluster-major) feed the next scatter.
template <int MODE>
__global__ __launch_bounds__(256) void assign_kernel(IterBufs b, const int* __restrict__ counts_in,
                                                     const int* __restrict__ cl_in,
                                                     const int* __restrict__ pos,
                                                     int* __restrict__ cl_out,
                                                     int* __restrict__ counts_out,
                                                     int* __restrict__ changed,
                                                     double* __restrict__ obj,
                                                     float* __restrict__ z_out,
                                                     float* __restrict__ D_out) {
  extern __shared__ double smem_d[];
  const int k = b.k, tid = threadIdx.x;
  double* zd = smem_d;                 // k
  float* zf = (float*)(zd + k);        // k
  float* sc = zf + k;                  // k
  int* hist = (int*)(sc + k);          // k

  for (int j = tid; j < k; j += 256) hist[j] = 0;
  // Loads that do not wait for z are issued first (clamped to a valid point
  // so they need no branch).
  const int64_t i = (int64_t)blockIdx.x * kBlk + tid;
  const bool valid = i < b.n;
  const int64_t iv = valid ? i : b.n - 1;
  const int cl_i = cl_in[iv];
  float dg = 0.f;
  int64_t ei = iv;  // column of E^T holding point i
  if (MODE == 1) {
    dg = b.diagK[iv];
    if (pos) ei = pos[iv];
  }
  const int cnt0 = (MODE == 1 && tid < k) ? counts_in[tid] : 0;
  if (MODE == 1) {
    // sum_{i in L_j} E(i, j) from the reduction's nzpart parts: for k <= 256,
    // 256/k threads per cluster each add a fixed run of parts, and the runs
    // are added in order (a short latency chain instead of nzpart loads)
    __shared__ double zrun[256];
    const int G = k <= 256 ? 256 / k : 1;
    if (k <= 256) {
      const int j = tid / G, g = tid % G;
      double s = 0.0;
      if (j < k) {
        const int per = (b.nzpart + G - 1) / G, lo = g * per, hi = min(b.nzpart, lo + per);
        const double* zp = b.zpart + (int64_t)j * b.nzpart;
        for (int x = lo; x < hi; x += 4) {  // four loads in flight, added in order
          double v[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) v[u] = zp[min(x + u, hi - 1)];
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (x + u < hi) s += v[u];
        }
      }
      zrun[tid] = s;
      __syncthreads();
    }
    for (int j = tid; j < k; j += 256) {
      const int c = j == tid ? cnt0 : counts_in[j];
      double zs = 0.0;
      if (c > 0) {
        if (k <= 256) {
          for (int g = 0; g < G; ++g) zs += zrun[j * G + g];
        } else {
          const double* zp = b.zpart + (int64_t)j * b.nzpart;
          for (int s = 0; s < b.nzpart; ++s) zs += zp[s];
        }
      }
      const double z = c > 0 ? zs / ((double)c * (double)c) : 0.0;
      zd[j] = c > 0 ? zs / (double)c : 0.0;  // |L_j| z_j
      zf[j] = (float)z;
      sc[j] = c > 0 ? -2.0f / (float)c : 0.f;
      if (blockIdx.x == 0 && z_out) z_out[j] = (float)z;
    }
  }
  __syncthreads();
  if (MODE == 1 && blockIdx.x == 0 && tid == 0 && obj) {
    double s = 0.0;
    for (int j = 0; j < k; ++j) s += zd[j];
    *obj = *b.trK - s;  // J(cl_in) = tr K - sum_j |L_j| z_j
  }

  int lab = 0, chg = 0;
  if (valid) {
    if (MODE == 0) {
      lab = cl_i;
      if (lab < 0 || lab >= k) {
        atomicOr(b.status, 1);
        lab = clamp_id(lab, k);
      }
    } else {
      float best = INFINITY;
      int arg = -1;
      for (int j0 = 0; j0 < k; j0 += 8) {
        // eight entries of E in flight (E^T has k rows, so the clamped reads
        // stay inside it); empty clusters are read but not used
        float ev[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) ev[u] = b.Et[(int64_t)min(j0 + u, k - 1) * b.ld + ei];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int j = j0 + u;
          if (j < k) {
            const float s = sc[j];
            float Dv = INFINITY;
            if (s != 0.f) {
              Dv = fmaf(s, ev[u], dg + zf[j]);
              if (arg < 0 || Dv < best) {
                best = Dv;
                arg = j;
              }
            }
            if (D_out) D_out[i * k + j] = Dv;
          }
        }
      }
      lab = arg < 0 ? 0 : arg;
      chg = (lab != clamp_id(cl_i, k));
      cl_out[i] = lab;
    }
    atomicAdd(&hist[lab], 1);
  }
  const int nchg = __syncthreads_count(chg);
  for (int j = tid; j < k; j += 256) {
    const int c = hist[j];
    b.hist[(int64_t)j * b.nblk + blockIdx.x] = c;
    if (c) atomicAdd(&counts_out[j], c);
  }
  if (MODE == 1 && tid == 0 && nchg && changed) atomicAdd(changed, nchg);
}

static size_t assign_smem(int k) { return (size_t)k * 20 + 64; }

// Points u < m, one per thread: D(u,j) = diag(u) - 2 E(u,j)/|L_j| + z_j for
// nonempty j (the full-step assign's formula, with z and the sizes given),
// lowest-index argmin; the new sizes are counted per workgroup in LDS.
// E(u, j) is read at E[u * s_pt + j * s_cl]: a panel's E^T in place
// (s_pt = 1, s_cl = ld) or a caller's E, point-major (s_pt = k, s_cl = 1).
__global__ __launch_bounds__(256) void cols_assign_kernel(const float* __restrict__ E, int64_t s_pt, int64_t s_cl,
                                                          const float* __restrict__ diag, int64_t m, int k,
                                                          const float* __restrict__ z,
                                                          const int* __restrict__ counts,
                                                          int* __restrict__ cl_out,
                                                          int* __restrict__ counts_out,
                                                          float* __restrict__ E_out) {
  extern __shared__ float psm[];
  const int tid = threadIdx.x;
  float* zf = psm;                // k
  float* sc = zf + k;             // k
  int* hist = (int*)(sc + k);     // k
  for (int j = tid; j < k; j += 256) {
    const int c = counts[j];
    zf[j] = z[j];
    sc[j] = c > 0 ? -2.0f / (float)c : 0.f;
    hist[j] = 0;
  }
  __syncthreads();
  const int64_t u = (int64_t)blockIdx.x * 256 + tid;
  if (u < m) {
    const float dg = diag[u];
    float best = INFINITY;
    int arg = -1;
    for (int j = 0; j < k; ++j) {
      const float e = E[u * s_pt + (int64_t)j * s_cl];
      if (E_out) E_out[u * k + j] = e;
      const float s = sc[j];
      if (s != 0.f) {
        const float Dv = fmaf(s, e, dg + zf[j]);
        if (arg < 0 || Dv < best) {
          best = Dv;
          arg = j;
        }
      }
    }
    const int lab = arg < 0 ? 0 : arg;
    cl_out[u] = lab;
    atomicAdd(&hist[lab], 1);
  }
  __syncthreads();
  for (int j = tid; j < k; j += 256)
    if (hist[j]) atomicAdd(&counts_out[j], hist[j]);
}

hipError_t launch_cols_assign(const float* E, int64_t s_pt, int64_t s_cl, const float* diag, int64_t m, int k,
                              const float* z, const int* counts, int* cl_out, int* counts_out, float* E_out,
                              hipStream_t s) {
  const unsigned grid = (unsigned)((m + 255) / 256);
  hipLaunchKernelGGL(cols_assign_kernel, dim3(grid), dim3(256), (size_t)k * 12, s, E, s_pt, s_cl, diag, m, k, z,
                     counts, cl_out, counts_out, E_out);
  return hipGetLastError();
}

hipError_t launch_panel_assign(const IterBufs& b, const float* z, const int* counts, int* cl_out,
                               int* counts_out, float* E_out, hipStream_t s) {
  return launch_cols_assign(b.Et, 1, b.ld, b.diagK + b.col0, b.ncol, b.k, z, counts, cl_out, counts_out, E_out, s);
}

// Workgroup g: points u in [1024 g, 1024 g + 1024) of a piece of m points
// (E point-major, m x k; ids cl): the piece's share of sum_{u in L_j} E(u, j)
// for each cluster j, in fp64 and a fixed order, at zpart[j * nz + g]; its
// cluster sizes added to counts; an id outside [0, k) sets bit 0 of status.
__global__ __launch_bounds__(256) void cols_zpart_kernel(const float* __restrict__ E, const int* __restrict__ cl,
                                                         int64_t m, int k, double* __restrict__ zpart, int nz,
                                                         int* __restrict__ counts, int* __restrict__ status) {
  extern __shared__ int zhist[];  // k
  __shared__ double red[4];
  const int tid = threadIdx.x;
  for (int j = tid; j < k; j += 256) zhist[j] = 0;
  __syncthreads();
  int jid[4];
  float ev[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int64_t u = (int64_t)blockIdx.x * 1024 + c * 256 + tid;
    jid[c] = -1;
    ev[c] = 0.f;
    if (u < m) {
      const int j = cl[u];
      if (j < 0 || j >= k) {
        atomicOr(status, 1);
      } else {
        jid[c] = j;
        ev[c] = E[u * k + j];
        atomicAdd(&zhist[j], 1);
      }
    }
  }
  __syncthreads();
  for (int j = tid; j < k; j += 256)
    if (zhist[j]) atomicAdd(&counts[j], zhist[j]);
  for (int j = 0; j < k; ++j) {
    double v = 0.0;
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (jid[c] == j) v += (double)ev[c];
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    if ((tid & 63) == 0) red[tid >> 6] = v;
    __syncthreads();
    if (tid == 0) zpart[(int64_t)j * nz + blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
    __syncthreads();
  }
}

hipError_t launch_cols_zpart(const float* E, const int* cl, int64_t m, int k, double* zpart, int nz, int* counts,
                             int* status, hipStream_t s) {
  const int64_t grid = (m + 1023) / 1024;
  if (m < 1 || grid > nz) return hipErrorInvalidValue;
  hipLaunchKernelGGL(cols_zpart_kernel, dim3((unsigned)grid), dim3(256), (size_t)k * 4, s, E, cl, m, k, zpart, nz,
                     counts, status);
  return hipGetLastError();
}

hipError_t launch_assign(int mode, const IterBufs& b, const int* counts_in, const int* cl_in,
                         const int* pos, int* cl_out, int* counts_out, int* changed, double* obj,
                         float* z_out, float* D_out, hipStream_t s) {
  dim3 grid((unsigned)b.nblk), block(256);
  const size_t sm = assign_smem(b.k);
  if (mode == 0)
    hipLaunchKernelGGL(assign_kernel<0>, grid, block, sm, s, b, counts_in, cl_in, pos, cl_out,
                       counts_out, changed, obj, z_out, D_out);
  else
    hipLaunchKernelGGL(assign_kernel<1>, grid, block, sm, s, b, counts_in, cl_in, pos, cl_out,
                       counts_out, changed, obj, z_out, D_out);
  return hipGetLastError();
}

// ----------------------------------------------------------------- scatter
//
// Stable counting sort of the points by cluster.  Point i of block blk goes to
//   off[c] + (members of c in blocks before blk) + (members of c in earlier
//   wavefronts of blk) + (members of c in earlier lanes of its wavefront),
// c = cl(i), from the per-block histograms of the previous kernel.  Each
// workgroup sums the histograms it needs itself.  Workgroup 0 also writes
// the SpMM chunk table (chunk q: cluster j, sorted positions [p0, p1), at
// most kChunk long) and clears this update's size and change counters.
__global__ __launch_bounds__(256) void scatter_kernel(IterBufs b, const int* __restrict__ cl,
                                                      const int* __restrict__ counts,
                                                      int* __restrict__ zero_counts,
                                                      int* __restrict__ zero_changed) {
  extern __shared__ int smem_i[];
  const int k = b.k, nb = b.nblk, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int blk = blockIdx.x;
  int* wc = smem_i;          // 4 x k: per-wavefront counts of each cluster
  int* offs = wc + 4 * k;    // k + 1: cluster offsets in the sorted order
  int* qf = offs + k + 1;    // k + 1: first chunk of each cluster
  int* basej = qf + k + 1;   // k: sorted position of this block's first member of j
  int* segsum = basej + k;   // 256
  int* cnt = segsum + 512;   // k: cluster sizes (after labs)

  const int64_t i = (int64_t)blk * kBlk + tid;
  const bool valid = i < b.n;
  const int lab = valid ? clamp_id(cl[i], k) : -1;
  for (int q = tid; q < 4 * k; q += 256) wc[q] = 0;
  for (int j = tid; j < k; j += 256) cnt[j] = counts[j];
  // members of each cluster in earlier blocks: for k <= 256, 256/k threads
  // per cluster each add a run of blocks (integers: any order is exact)
  const int G = k <= 256 ? 256 / k : 1, jg = tid / G, g = tid % G;
  if (k <= 256) {
    const int seg = (blk + G - 1) / G, lo = g * seg, hi = (lo + seg < blk) ? lo + seg : blk;
    int s = 0;
    if (jg < k) {
      const int* hj = b.hist + (int64_t)jg * nb;
      for (int bb = lo; bb < hi; bb += 4) {  // four loads in flight
        int v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = hj[min(bb + u, hi - 1)];
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (bb + u < hi) s += v[u];
      }
    }
    segsum[tid] = s;
  }
  __syncthreads();
  if (tid == 0) {
    int o = 0, q = 0;
    for (int j = 0; j < k; ++j) {
      const int c = cnt[j];
      offs[j] = o;
      qf[j] = q;
      o += c;
      q += (c + b.chunk_len - 1) / b.chunk_len;
    }
    offs[k] = o;
    qf[k] = q;
  }
  __syncthreads();
  if (k <= 256) {
    if (jg < k && g == 0) {
      int run = offs[jg];
      for (int gg = 0; gg < G; ++gg) run += segsum[jg * G + gg];
      basej[jg] = run;
    }
  } else {
    for (int j = tid; j < k; j += 256) {
      int run = offs[j];
      for (int bb = 0; bb < blk; ++bb) run += b.hist[(int64_t)j * nb + bb];
      basej[j] = run;
    }
  }
  if (blk == 0) {
    if (zero_counts)
      for (int j = tid; j < k; j += 256) zero_counts[j] = 0;
    if (zero_changed && tid == 0) *zero_changed = 0;
    for (int j = tid; j <= k; j += 256) {
      b.off[j] = offs[j];
      b.qfirst[j] = qf[j];
    }
    if (tid == 0) *b.nchunks = qf[k];
    for (int q = tid; q < qf[k]; q += 256) {
      int lo = 0, hi = k - 1;  // last j with qf[j] <= q
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (qf[mid] <= q) lo = mid;
        else hi = mid - 1;
      }
      const int p0 = offs[lo] + (q - qf[lo]) * b.chunk_len, end = offs[lo + 1];
      b.chunk_j[q] = lo;
      b.chunk_p0[q] = p0;
      b.chunk_p1[q] = (p0 + b.chunk_len < end) ? p0 + b.chunk_len : end;
    }
    // packed K: the chunk-major member table ends each cluster's last chunk
    // and starts each unused chunk with -1 (the members are written below)
    if (b.crow) {
      const int cl = b.chunk_len;
      for (int j = 0; j < k; ++j)
        for (int64_t x = (int64_t)qf[j] * cl + (offs[j + 1] - offs[j]) + tid; x < (int64_t)qf[j + 1] * cl; x += 256)
          b.crow[x] = -1;
      for (int q = qf[k] + tid; q < b.qmax; q += 256) b.crow[(int64_t)q * cl] = -1;
    }
  }

  int* labs = segsum + 256;  // this block's 256 ids (-1 past n), for the packed one-hot masks
  labs[tid] = lab;
  int rank = 0;
  unsigned long long todo = __ballot(valid);
  while (todo) {
    const int leader = __ffsll((long long)todo) - 1;
    const int L = __shfl(lab, leader, 64);
    const unsigned long long m = __ballot(lab == L);
    if (lab == L) rank = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == leader) wc[w * k + L] = __popcll(m);
    todo &= ~m;
  }
  __syncthreads();
  if (valid) {
    int r = basej[lab] + rank;
    for (int ww = 0; ww < w; ++ww) r += wc[ww * k + lab];
    b.perm[r] = (int)i;
    b.pos[i] = r;
    // packed K: the first member of a chunk (members are in index order)
    // fixes the chunk's first stored column
    const int rel = r - offs[lab];
    if (b.chunk_c0 && rel % b.chunk_len == 0)
      b.chunk_c0[qf[lab] + rel / b.chunk_len] = (int)(i / kTile) * kTile;
    if (b.crow) b.crow[(int64_t)qf[lab] * b.chunk_len + rel] = (int)i;
  }
  // packed K: the one-hot bits of this block's two column tiles, once per
  // update (the SpMM reads them instead of the ids)
  if (b.mskg) {
    const int per_tile = b.nlb * 64;
    for (int t = tid; t < 2 * per_tile; t += 256) {
      const int half = t / per_tile, rem = t % per_tile;
      const int J = 2 * blk + half;
      if ((int64_t)J * kTile >= b.n) continue;
      const int nb = rem >> 6, kk = (rem >> 4) & 3, want = 16 * nb + (rem & 15);
      const int* lt = labs + half * kTile + 4 * kk;
      unsigned m = 0;
#pragma unroll
      for (int g = 0; g < 8; ++g)
#pragma unroll
        for (int e = 0; e < 4; ++e) m |= (unsigned)(lt[16 * g + e] == want) << (4 * g + e);
      b.mskg[(int64_t)J * per_tile + rem] = m;
    }
  }
}

hipError_t launch_scatter(const IterBufs& b, const int* cl, const int* counts, int* zero_counts,
                          int* zero_changed, hipStream_t s) {
  const size_t sm = (size_t)(8 * b.k + 2 + 512) * sizeof(int);
  hipLaunchKernelGGL(scatter_kernel, dim3((unsigned)b.nblk), dim3(256), sm, s, b, cl, counts,
                     zero_counts, zero_changed);
  return hipGetLastError();
}

// ----------------------------------------------------------------- SpMM
//
// Workgroup (stripe, q): columns [stripe*1024, +1024) of the rows listed in
// chunk q (one cluster j, at most kChunk rows in sorted order).  Each lane keeps
// one float4 accumulator; rows are summed in sorted order with non-temporal
// 16-byte loads (K has no reuse within an update) and the chunk's sum goes
// to P[q].  A second kernel adds the chunks of each cluster in chunk order;
// the kernel boundary makes the partial sums visible across XCDs without a
// device-scope fence per workgroup, which costs more than half the bandwidth.
// KT: float, or binary16 with row r's entries divided by kw[r] (kw null: 1);
// binary16 rows are read 4 entries (8 bytes) per lane, widened and scaled.
template <typename KT>
__global__ __launch_bounds__(256) void spmm_onehot_kernel(const KT* __restrict__ K, IterBufs b) {
  constexpr bool kHalf = sizeof(KT) == 2;
  const int ns = b.nstripes;
  const int stripe = (int)(blockIdx.x % (unsigned)ns);
  const int q = (int)(blockIdx.x / (unsigned)ns);
  if (q >= *b.nchunks) return;
  const int p0 = b.chunk_p0[q], p1 = b.chunk_p1[q];
  const int tid = threadIdx.x;
  __shared__ int rows[kChunk];
  __shared__ float rw[kHalf ? kChunk : 1];
  for (int p = p0 + tid; p < p1; p += 256) {
    const int r = b.perm[p];
    rows[p - p0] = r;
    if (kHalf) rw[p - p0] = b.kw ? b.kw[r] : 1.f;
  }
  __syncthreads();

  const int64_t ld = b.ld;
  const int64_t col = (int64_t)stripe * kStripe + tid * 4;
  if (col >= ld) return;
  f4 acc = {0.f, 0.f, 0.f, 0.f};
  const int nr = p1 - p0;
  const KT* base = K + col;
  auto row = [&](int r) {  // row r of the chunk at this lane's 4 columns
    if (kHalf) {
      const h4 v = __builtin_nontemporal_load((const h4*)(base + (int64_t)rows[r] * ld));
      return __builtin_convertvector(v, f4) * rw[r];
    } else {
      return (f4)__builtin_nontemporal_load((const f4*)(base + (int64_t)rows[r] * ld));
    }
  };
  int r = 0;
  for (; r + 8 <= nr; r += 8) {
    f4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = row(r + u);
#pragma unroll
    for (int u = 0; u < 8; ++u) acc += v[u];
  }
  for (; r < nr; ++r) acc += row(r);
  *(f4*)(b.P + (int64_t)q * ld + col) = acc;
}

// Workgroup (stripe, j): E^T(j, stripe) = sum of cluster j's chunk partials in
// chunk order, and the stripe's share of sum_{i in L_j} E(i, j) (fp64) for z_j.
__global__ __launch_bounds__(256) void spmm_reduce_kernel(IterBufs b, const int* __restrict__ cl) {
  const int ns = b.nstripes;
  const int stripe = (int)(blockIdx.x % (unsigned)ns);
  const int j = (int)(blockIdx.x / (unsigned)ns);
  const int qa = b.qfirst[j], qb = b.qfirst[j + 1];
  if (qa == qb) return;  // empty cluster: E^T(j, .) and z_j are never read
  const int tid = threadIdx.x;
  __shared__ double red[4];
  const int64_t ld = b.ld;
  const int64_t col = (int64_t)stripe * kStripe + tid * 4;
  double zs = 0.0;
  if (col < ld) {
    f4 e = *(const f4*)(b.P + (int64_t)qa * ld + col);
    for (int q = qa + 1; q < qb; ++q) e += *(const f4*)(b.P + (int64_t)q * ld + col);
    *(f4*)(b.Et + (int64_t)j * ld + col) = e;
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (col + c < b.ncol && cl[b.col0 + col + c] == j) zs += (double)e[c];
  }
  for (int off = 32; off > 0; off >>= 1) zs += __shfl_xor(zs, off, 64);
  if ((tid & 63) == 0) red[tid >> 6] = zs;
  __syncthreads();
  if (tid == 0) b.zpart[(int64_t)j * ns + stripe] = (red[0] + red[1]) + (red[2] + red[3]);
}

hipError_t launch_spmm_onehot(const void* K, const IterBufs& b, hipStream_t s) {
  const long long grid = (long long)b.nstripes * b.qmax;
  if (b.kf16)
    hipLaunchKernelGGL(spmm_onehot_kernel<half_t>, dim3((unsigned)grid), dim3(256), 0, s, (const half_t*)K, b);
  else
    hipLaunchKernelGGL(spmm_onehot_kernel<float>, dim3((unsigned)grid), dim3(256), 0, s, (const float*)K, b);
  return hipGetLastError();
}

// Rows r0 .. r1-1 of a full binary16 K, widened and scaled back to fp32.
__global__ __launch_bounds__(256) void rows_f16_kernel(const half_t* __restrict__ K, const float* __restrict__ kw,
                                                       int64_t n, int64_t ld, int64_t r0, int64_t r1,
                                                       float* __restrict__ out) {
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (c >= n) return;
  for (int64_t r = r0 + blockIdx.y; r < r1; r += gridDim.y)
    out[(r - r0) * n + c] = (float)K[r * ld + c] * (kw ? kw[r] : 1.f);
}

hipError_t launch_rows_f16(const half_t* K, const float* kw, int64_t n, int64_t ld, int64_t r0, int64_t r1,
                           float* out, hipStream_t s) {
  const unsigned gy = (unsigned)std::min<int64_t>(r1 - r0, 65535);
  hipLaunchKernelGGL(rows_f16_kernel, dim3((unsigned)((n + 255) / 256), gy), dim3(256), 0, s, K, kw, n, ld, r0,
                     r1, out);
  return hipGetLastError();
}

hipError_t launch_spmm_reduce(const IterBufs& b, const int* cl, hipStream_t s) {
  hipLaunchKernelGGL(spmm_reduce_kernel, dim3((unsigned)(b.nstripes * b.k)), dim3(256), 0, s, b, cl);
  return hipGetLastError();
}

// Workgroup (stripe, j): a block's partial E(u, j), the sum over its rows in
// cluster j of K(row, c0 + u) (cluster j's chunk partials added in chunk
// order; 0 where none of the block's rows is in cluster j), stored
// point-major at E_out[u * k + j] for u < ncol.
__global__ __launch_bounds__(256) void block_out_kernel(IterBufs b, float* __restrict__ E_out) {
  const int ns = b.nstripes;
  const int stripe = (int)(blockIdx.x % (unsigned)ns);
  const int j = (int)(blockIdx.x / (unsigned)ns);
  const int qa = b.qfirst[j], qb = b.qfirst[j + 1];
  const int64_t ld = b.ld;
  const int64_t col = (int64_t)stripe * kStripe + threadIdx.x * 4;
  if (col >= b.ncol) return;
  f4 e = {0.f, 0.f, 0.f, 0.f};
  for (int q = qa; q < qb; ++q) e += *(const f4*)(b.P + (int64_t)q * ld + col);
#pragma unroll
  for (int c = 0; c < 4; ++c)
    if (col + c < b.ncol) E_out[(col + c) * b.k + j] = e[c];
}

hipError_t launch_block_out(const IterBufs& b, float* E_out, hipStream_t s) {
  hipLaunchKernelGGL(block_out_kernel, dim3((unsigned)(b.nstripes * b.k)), dim3(256), 0, s, b, E_out);
  return hipGetLastError();
}

// E (n x k, row-major) from E^T; empty clusters read as 0.
__global__ void et_to_e_kernel(IterBufs b, const int* __restrict__ counts, const int* __restrict__ pos,
                               float* __restrict__ E) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= b.n * b.k) return;
  const int64_t i = t / b.k;
  const int j = (int)(t % b.k);
  const int64_t ei = pos ? (int64_t)pos[i] : i;
  E[t] = counts[j] > 0 ? b.Et[(int64_t)j * b.ld + ei] : 0.f;
}

hipError_t launch_et_to_e(const IterBufs& b, const int* counts, const int* pos, float* E,
                          hipStream_t s) {
  const int64_t tot = b.n * b.k;
  hipLaunchKernelGGL(et_to_e_kernel, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, b,
                     counts, pos, E);
  return hipGetLastError();
}

}  // namespace kkm
