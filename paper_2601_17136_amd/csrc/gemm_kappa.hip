// K = kappa(X X^T): the Gram GEMM of Eq. 1 with the kernel function of Eq. 2
// (or the linear / Gaussian kernel) applied in the epilogue.
//
// B = X X^T is symmetric, so only tiles (I, J) with I <= J of the 128 x 128
// tiling are computed.  Full storage keeps an off-diagonal tile twice, as
// itself and, transposed through LDS, as tile (J, I); packed storage keeps
// only the computed tiles (the upper block triangle, see packed_row).  The
// product runs on the fp32 matrix cores (v_mfma_f32_32x32x2_f32).  Each
// 256-thread workgroup owns one tile, each wavefront a 64 x 64 quarter of it
// (2 x 2 MFMA blocks of 32 x 32).
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

// Row scales of binary16 storage: |x_i . x_j| <= |x_i| max_m |x_m|
// (Cauchy-Schwarz), so kw[i] bounds every |K(i, j)|; 1 for a zero row.
__global__ void row_scales_kernel(const float* __restrict__ nrm, const unsigned* __restrict__ maxnrm_bits,
                                  int64_t n, KappaParams kp, float* __restrict__ kw) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float dot = sqrtf(nrm[i] * __uint_as_float(*maxnrm_bits));
  float w = dot;
  if (kp.kind == POLY) {
    const float t = fmaf(fabsf(kp.gamma), dot, fabsf(kp.coef0));
    w = 1.f;
    for (int e = 0; e < kp.degree; ++e) w *= t;
  }
  kw[i] = w > 0.f ? w : 1.f;
}

hipError_t launch_row_scales(const float* nrm, const unsigned* maxnrm_bits, int64_t n, const KappaParams& kp,
                             float* kw, hipStream_t s) {
  hipLaunchKernelGGL(row_scales_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, nrm, maxnrm_bits, n,
                     kp, kw);
  return hipGetLastError();
}

// Four workgroups per CU (40 KB of LDS each): while some run their store
// epilogue, others keep the matrix cores busy.  KT is the storage type of K
// (float, or binary16 with entry (i, j) divided by kw[i]).
// PANEL: the block K[r0:r1, c0 : c0 + ld) of one GPU's share (r0 and c0
// multiples of kTile, columns past c1 stored as 0): every tile (I, J) in
// the block, each stored once at (i - r0, j - c0); nt counts the block's
// column tiles there, and T = its row tiles x nt.
template <int KIND, typename KT, bool PANEL>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void gemm_kappa_kernel(
    const float* __restrict__ Xp, const float* __restrict__ nrm,
    const unsigned* __restrict__ maxnrm_bits, int64_t n, int d_pad, int64_t ld, bool packed,
    int64_t nt, int64_t T, int64_t r0, int64_t r1, int64_t c0, int64_t c1, KappaParams kp,
    KT* __restrict__ K, const float* __restrict__ kw, float* __restrict__ diagK,
    int2* __restrict__ fix_list, unsigned long long* __restrict__ fix_count, long long seg_cap) {
  constexpr bool kHalf = sizeof(KT) == 2;
  __shared__ __attribute__((aligned(16))) float lds[kLdsFloats];
  // No Gaussian entry can need the fix-up unless the largest norms allow it.
  const bool may_fix = KIND == GAUSS && gauss_needs_fix(1.f, __uint_as_float(*maxnrm_bits),
                                                         __uint_as_float(*maxnrm_bits), kp);

  // Workgroup b runs on XCD b % 8.  Give each XCD a contiguous run of tiles
  // so that concurrent workgroups of one XCD share row block I in its L2.
  const int64_t b = blockIdx.x;
  const int64_t per = T >> 3, rem = T & 7, x = b & 7;
  const int64_t t = x * per + (x < rem ? x : rem) + (b >> 3);
  int64_t I, J;
  if (PANEL) {
    I = r0 / kTile + t / nt;
    J = c0 / kTile + t % nt;
  } else {
    triangle_tile(t, nt, I, J);
  }
  const int64_t row0 = I * kTile, col0 = J * kTile;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l32 = lane & 31, h = lane >> 5;

  floatx16 acc[2][2];
  mma_tile(Xp + row0 * d_pad, Xp + col0 * d_pad, d_pad, lds, acc);

  // ---- epilogue: acc[bi][bj][r] is B(i, j) with
  //      i = row0 + wm*64 + bi*32 + 8*(r/4) + 4*h + r%4,  j = col0 + wn*64 + bj*32 + l32
  // Rows 8q + 4h .. 8q + 4h + 3 of a 32-row block are consecutive, so their
  // norms come in one 16-byte load.
  // The Gaussian works on the norms scaled by c = -gamma log2(e) (gauss_scaled).
  const float cg = kp.neg_g_log2e;
  float cnj[2] = {0.f, 0.f};
  const float* nrow = nrm + row0 + wm * 64 + 4 * h;
  if (KIND == GAUSS) {
    cnj[0] = cg * nrm[col0 + wn * 64 + l32];
    cnj[1] = cg * nrm[col0 + wn * 64 + 32 + l32];
  }
  bool flagged = false;  // some entry of this lane may need the fix-up
#pragma unroll
  for (int bi = 0; bi < 2; ++bi) {
    // u = c|x_i|^2 + c|x_j|^2 rounds the same for (i, j) and (j, i) only
    // if the products are not fused into the sum
#pragma clang fp contract(off)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float4 n4 = {0.f, 0.f, 0.f, 0.f};
      if (KIND == GAUSS) n4 = *(const float4*)(nrow + bi * 32 + 8 * q);
      const float cn[4] = {cg * n4.x, cg * n4.y, cg * n4.z, cg * n4.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
#pragma unroll
        for (int bj = 0; bj < 2; ++bj) {
          float v;
          if (KIND == GAUSS) {
            const float u = cn[e] + cnj[bj];
            v = gauss_scaled(acc[bi][bj][4 * q + e], u, kp);
            if (may_fix) flagged |= gauss_needs_fix_scaled(v, u, kp);
          } else {
            v = kappa<KIND>(acc[bi][bj][4 * q + e], 0.f, 0.f, kp);
          }
          acc[bi][bj][4 * q + e] = v;
        }
      }
    }
  }
  // The diagonal: only tiles I == J hold it, in the blocks bi == bj of the
  // waves with wm == wn (il == jl there means 8*(r/4) + 4h + r%4 == l32).
  if (I == J && wm == wn) {
#pragma unroll
    for (int bi = 0; bi < 2; ++bi) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        if (8 * (r >> 2) + 4 * h + (r & 3) == l32) {
          const int64_t gi = row0 + wm * 64 + bi * 32 + l32;
          float v = acc[bi][bi][r];
          if (KIND == GAUSS) v = 1.f;  // exp(0): exact, whatever B(i,i) rounded to
          acc[bi][bi][r] = v;
          if (gi < n) diagK[gi] = v;
        }
      }
    }
  }
  // Gaussian entries to recompute: the estimate above is taken for every
  // entry; only where some lane flagged one are the listed pairs formed.
  // The square layouts list each pair once (i < j) for both of its entries;
  // a panel lists every entry it stores.  Each lane marks its listed
  // entries in a 64-bit mask (entry g = ((bi*4 + q)*4 + e)*2 + bj); a scan
  // of the lanes' counts and one atomic per wavefront give the slots.  (A
  // returning atomic per group of 64 entries left the wavefront waiting on
  // one round trip per group.)  The test repeats the estimate above with
  // the same operands.
  if (KIND == GAUSS && may_fix && __ballot(flagged)) {
    const int seg = (int)(blockIdx.x % kFixSegs);
    unsigned mlo = 0u, mhi = 0u;
#pragma unroll
    for (int bi = 0; bi < 2; ++bi) {
#pragma clang fp contract(off)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 n4 = *(const float4*)(nrow + bi * 32 + 8 * q);
        const float cn[4] = {cg * n4.x, cg * n4.y, cg * n4.z, cg * n4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int64_t gi = row0 + wm * 64 + bi * 32 + 8 * q + 4 * h + e;
#pragma unroll
          for (int bj = 0; bj < 2; ++bj) {
            const int64_t gj = col0 + wn * 64 + bj * 32 + l32;
            const bool f = (PANEL ? (gi != gj && gi < r1 && gj < c1) : (gi < gj && gj < n)) &&
                           gauss_needs_fix_scaled(acc[bi][bj][4 * q + e], cn[e] + cnj[bj], kp);
            const int g = ((bi * 4 + q) * 4 + e) * 2 + bj;
            if (g < 32) mlo |= f ? 1u << g : 0u;
            else mhi |= f ? 1u << (g - 32) : 0u;
          }
        }
      }
    }
    const unsigned cnt = (unsigned)(__popc(mlo) + __popc(mhi));
    unsigned pre = cnt;  // inclusive scan over the lanes
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const unsigned v = __shfl_up(pre, o, 64);
      if (lane >= o) pre += v;
    }
    const unsigned total = __shfl(pre, 63, 64);
    unsigned long long base = 0;
    if (lane == 0 && total) base = atomicAdd(fix_count + seg, (unsigned long long)total);
    base = __shfl(base, 0, 64) + (pre - cnt);
    while (mlo | mhi) {
      const int g = mlo ? __ffs(mlo) - 1 : 32 + __ffs(mhi) - 1;
      if (g < 32) mlo &= mlo - 1u;
      else mhi &= mhi - 1u;
      const int bj = g & 1, e = (g >> 1) & 3, q = (g >> 3) & 3, bi = g >> 5;
      const int64_t gi = row0 + wm * 64 + bi * 32 + 8 * q + 4 * h + e;
      const int64_t gj = col0 + wn * 64 + bj * 32 + l32;
      if (base < (unsigned long long)seg_cap)
        fix_list[(int64_t)seg * seg_cap + (int64_t)base] = make_int2((int)gi, (int)gj);
      ++base;
    }
  }

  // ---- stores of tile (I, J).  The rows of a tile lie at a fixed stride S
  //      in every layout (packed: ld - row0), so entry (il, jl) of the tile
  //      is at Kb + il S + jl.  Non-temporal: K is not read again here.
  //      fp32 goes straight from the MFMA layout: each instruction writes
  //      rows il and il + 4, 32 consecutive floats (128 bytes) each, and
  //      the address is a uniform base plus a per-lane 32-bit offset fixed
  //      for the tile (S < kMaxKStride keeps it below 2^32 bytes; the
  //      launchers and the panel and block builds check).  Binary16 is
  //      staged through LDS instead,
  //      so each instruction writes one row's 128 contiguous bytes.
  // Columns j < clim hold entries, clim <= j < cend hold 0 (the padding of
  // a row), and j >= cend lie past the row's end.
  KT* Kb;
  int64_t S, rlim, clim, cend;
  if (PANEL) {
    Kb = K + (row0 - r0) * ld + (col0 - c0);
    S = ld;
    rlim = r1;
    clim = c1;
    cend = c0 + ld;
  } else {
    Kb = K + (packed ? packed_row(row0, ld) : row0 * ld) + col0;
    S = packed ? ld - row0 : ld;
    rlim = n;
    clim = n;
    cend = ld;
  }
  float* Tw = lds + wave * (32 * 65);
  if (!kHalf) {
    // row il = bi*32 + 8(r/4) + (r%4) + 4h: the uniform part gives each
    // row's base address, the rest is one per-lane byte offset for all rows
    const unsigned lane_b = ((unsigned)(wm * 64 + 4 * h) * (unsigned)S + (unsigned)(wn * 64 + l32)) * 4u;
    char* const Kc = (char*)Kb;
    const bool full = row0 + kTile <= rlim && col0 + kTile <= clim;
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int iu = bi * 32 + 8 * (r >> 2) + (r & 3);
        char* const rowp = Kc + (size_t)iu * (size_t)S * 4u;
        float v0 = acc[bi][0][r], v1 = acc[bi][1][r];
        if (full) {
          __builtin_nontemporal_store(v0, (float*)(rowp + lane_b));
          __builtin_nontemporal_store(v1, (float*)(rowp + lane_b + 128u));
          continue;
        }
        // the last row or column block: rows past rlim are not stored;
        // columns past clim hold 0 up to the row's end (ld), none beyond
        if (row0 + wm * 64 + 4 * h + iu >= rlim) continue;
        const int64_t j0 = col0 + wn * 64 + l32, j1 = j0 + 32;
        if (j0 < cend) __builtin_nontemporal_store(j0 < clim ? v0 : 0.f, (float*)(rowp + lane_b));
        if (j1 < cend) __builtin_nontemporal_store(j1 < clim ? v1 : 0.f, (float*)(rowp + lane_b + 128u));
      }
  } else {
    auto put = [&](int64_t gi, float v, KT* dst) {
      const float inv = kw ? 1.f / kw[gi] : 1.f;
      __builtin_nontemporal_store((KT)(v * inv), dst);
    };
#pragma unroll
    for (int bi = 0; bi < 2; ++bi) {
#pragma unroll
      for (int bj = 0; bj < 2; ++bj)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          Tw[(8 * (r >> 2) + 4 * h + (r & 3)) * 65 + bj * 32 + l32] = acc[bi][bj][r];
      __syncthreads();
      const int jl = wn * 64 + lane;
      const int il0 = wm * 64 + bi * 32;
      const int nrows = (int)min<int64_t>(32, rlim - (row0 + il0));
      const bool col_val = col0 + jl < clim;
      KT* dst = Kb + il0 * S + jl;
      if (col0 + jl < cend) {
        if (nrows >= 32) {
#pragma unroll
          for (int rr = 0; rr < 32; ++rr) put(row0 + il0 + rr, col_val ? Tw[rr * 65 + lane] : 0.f, dst + rr * S);
        } else {
          for (int rr = 0; rr < nrows; ++rr) put(row0 + il0 + rr, col_val ? Tw[rr * 65 + lane] : 0.f, dst + rr * S);
        }
      }
      __syncthreads();
    }
  }
  if (!PANEL && I != J && !packed) {
#pragma unroll
    for (int bj = 0; bj < 2; ++bj) {  // tile (J, I): rows j, columns i
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          Tw[l32 * 65 + bi * 32 + 8 * (r >> 2) + 4 * h + (r & 3)] = acc[bi][bj][r];
      __syncthreads();
      const int64_t gj = row0 + wm * 64 + lane;  // I < J, so gj < n
      const int64_t gi0 = col0 + wn * 64 + bj * 32;
      const int nrows = (int)min<int64_t>(32, n - gi0);
      KT* dst = K + gi0 * ld + gj;
      auto put = [&](int rr) {
        const float v = Tw[rr * 65 + lane];
        if (kHalf) __builtin_nontemporal_store((KT)(v * (kw ? 1.f / kw[gi0 + rr] : 1.f)), dst + rr * ld);
        else __builtin_nontemporal_store((KT)v, dst + rr * ld);
      };
      if (nrows >= 32) {
#pragma unroll
        for (int rr = 0; rr < 32; ++rr) put(rr);
      } else {
        for (int rr = 0; rr < nrows; ++rr) put(rr);
      }
      __syncthreads();
    }
  }
}

// ---- Small widths (d_pad <= kRegMaxDpad, fp32 storage, the square layouts):
// the build as a sweep.  A workgroup owns row block I and a segment of
// column tiles J >= I (the on-the-fly sweep's work items): the block's rows
// are staged in LDS once, each wavefront loads its 64 columns of tile J into
// registers (mma_rows_lds), and nothing ties the four wavefronts together
// inside the sweep: the epilogue is gemm_kappa_kernel's (kappa, the diagonal,
// the fix-up listing, stores straight from the MFMA layout), and the mirror
// of a full-storage tile goes through the wavefront's own LDS tile, ordered
// within the wavefront.  Two workgroups per CU, so every SIMD holds two
// independent wavefronts.
__device__ __host__ inline int sweep_seg_begin(int s, int nt, int nseg) { return (int)((int64_t)s * nt / nseg); }

int build_sweep_segments(int64_t n) {
  const int nt = (int)((n + kTile - 1) / kTile);
  int nseg = (8192 + nt - 1) / nt;  // ~4096 work items right of the diagonal
  if (nseg > nt) nseg = nt;
  if (nseg > 64) nseg = 64;
  return nseg < 1 ? 1 : nseg;
}

template <int KIND, int HP, bool PACKED>
__global__ __launch_bounds__(256, 2) void gemm_kappa_sweep_kernel(
    const float* __restrict__ Xp, const float* __restrict__ nrm, const unsigned* __restrict__ maxnrm_bits,
    int64_t n, int64_t ld, int nt, int nseg, KappaParams kp, float* __restrict__ K,
    float* __restrict__ diagK, int2* __restrict__ fix_list, unsigned long long* __restrict__ fix_count,
    long long seg_cap, const float* __restrict__ bmax) {
  constexpr int d_pad = 2 * HP, ldsA = 2 * HP + 4;
  __shared__ __attribute__((aligned(16))) float As[kTile * ldsA];
  __shared__ float Tm[PACKED ? 1 : 4 * 32 * 65];  // per wavefront: a 32 x 64 block transposed (full storage)
  __shared__ __attribute__((aligned(16))) float Ns[kTile];  // Gaussian: the block's squared norms times cg
  // work items (segment s, row block I < sweep_seg_begin(s+1)), segment-major
  int s = 0;
  int64_t first = 0;
  while (s + 1 < nseg && first + sweep_seg_begin(s + 1, nt, nseg) <= (int64_t)blockIdx.x) {
    first += sweep_seg_begin(s + 1, nt, nseg);
    ++s;
  }
  const int I = (int)((int64_t)blockIdx.x - first);
  const int sb = sweep_seg_begin(s, nt, nseg), se = sweep_seg_begin(s + 1, nt, nseg);
  if (I >= se) return;
  const int jt0 = sb > I ? sb : I, jt1 = se;
  const int64_t row0 = (int64_t)I * kTile;
  const bool may_fix = KIND == GAUSS && gauss_needs_fix(1.f, __uint_as_float(*maxnrm_bits),
                                                         __uint_as_float(*maxnrm_bits), kp);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, l32 = lane & 31, h = lane >> 5;
  const float cg = kp.neg_g_log2e;
  for (int f = tid; f < kTile * (HP / 2); f += 256) {  // the block's rows (zero padded past n)
    const int r = f / (HP / 2), c = f % (HP / 2);
    *(float4*)(As + r * ldsA + 4 * c) = *(const float4*)(Xp + (row0 + r) * d_pad + 4 * c);
  }
  if (KIND == GAUSS && tid < kTile) Ns[tid] = cg * nrm[row0 + tid];  // nrm is zero past n
  __syncthreads();
  const float* const Aw = As + wm * 64 * ldsA;
  float* const Tw = Tm + wave * (32 * 65);
  const float* const nrow = Ns + wm * 64 + 4 * h;  // this lane's rows' cg * |x|^2, from LDS
  const int64_t S = PACKED ? ld - row0 : ld;  // row stride of the block's stored rows
  float* const Kr = K + (PACKED ? packed_row(row0, ld) : row0 * ld);
  const unsigned lane_b = ((unsigned)(wm * 64 + 4 * h) * (unsigned)S + (unsigned)(wn * 64 + l32)) * 4u;

  // Tile J's column operands and (Gaussian) column norms.  They are loaded
  // for the next tile before this tile's stores are issued: loads and stores
  // share one in-order completion counter, so a load issued after the stores
  // would make the next tile's products wait for the stores to drain.  The
  // rows' norms come from LDS for the same reason.
  float b[2][HP];
  float nj[2] = {0.f, 0.f};  // the columns' squared norms (scaled where used, so nothing waits here)
  auto fetch = [&](int J, int q) {  // column block q (32 columns) of tile J
    const int64_t c = (int64_t)J * kTile + wn * 64 + q * 32 + l32;
    load_operand<HP>(Xp, c, d_pad, h, b[q]);
    if (KIND == GAUSS) nj[q] = nrm[c];
  };
  if (jt0 < jt1) {
    fetch(jt0, 0);
    fetch(jt0, 1);
  }

  for (int J = jt0; J < jt1; ++J) {
    const int64_t col0 = (int64_t)J * kTile;
    floatx16 acc[2][2];
    mma_rows_lds<HP>(Aw, b[0], acc[0][0], acc[1][0], l32, h);
    mma_rows_lds<HP>(Aw, b[1], acc[0][1], acc[1][1], l32, h);
    __builtin_amdgcn_sched_barrier(0);

    // kappa, as in gemm_kappa_kernel, with the fix-up estimate kept as one
    // running minimum of u v per lane, and taken only where the two blocks'
    // largest squared norms allow an entry of the tile to qualify
    float cnj[2] = {0.f, 0.f};
    if (KIND == GAUSS) {
      cnj[0] = cg * nj[0];
      cnj[1] = cg * nj[1];
    }
    const bool tile_fix = KIND == GAUSS && may_fix && gauss_needs_fix(1.f, bmax[I], bmax[J], kp);
    float umin = 0.f;
    auto kpass = [&](bool est) {
#pragma unroll
      for (int bi = 0; bi < 2; ++bi) {
#pragma clang fp contract(off)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float4 n4 = {0.f, 0.f, 0.f, 0.f};
          if (KIND == GAUSS) n4 = *(const float4*)(nrow + bi * 32 + 8 * q);
          const float cn[4] = {n4.x, n4.y, n4.z, n4.w};
#pragma unroll
          for (int e = 0; e < 4; ++e)
#pragma unroll
            for (int bj = 0; bj < 2; ++bj) {
              float v;
              if (KIND == GAUSS) {
                const float u = cn[e] + cnj[bj];
                v = gauss_scaled(acc[bi][bj][4 * q + e], u, kp);
                if (est) umin = fminf(umin, u * v);
              } else {
                v = kappa<KIND>(acc[bi][bj][4 * q + e], 0.f, 0.f, kp);
              }
              acc[bi][bj][4 * q + e] = v;
            }
        }
      }
    };
    if (tile_fix) kpass(true);
    else kpass(false);
    if (J == I && wm == wn) {  // the diagonal
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (8 * (r >> 2) + 4 * h + (r & 3) == l32) {
            const int64_t gi = row0 + wm * 64 + bi * 32 + l32;
            float v = acc[bi][bi][r];
            if (KIND == GAUSS) v = 1.f;
            acc[bi][bi][r] = v;
            if (gi < n) diagK[gi] = v;
          }
    }
    if (KIND == GAUSS && tile_fix && __ballot(umin < kp.fix_uthr)) {  // the listing, as in gemm_kappa_kernel
      const int seg = (int)(blockIdx.x % kFixSegs);
      unsigned mlo = 0u, mhi = 0u;
#pragma unroll
      for (int bi = 0; bi < 2; ++bi) {
#pragma clang fp contract(off)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 n4 = *(const float4*)(nrow + bi * 32 + 8 * q);
          const float cn[4] = {n4.x, n4.y, n4.z, n4.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int64_t gi = row0 + wm * 64 + bi * 32 + 8 * q + 4 * h + e;
#pragma unroll
            for (int bj = 0; bj < 2; ++bj) {
              const int64_t gj = col0 + wn * 64 + bj * 32 + l32;
              const bool f = gi < gj && gj < n && gauss_needs_fix_scaled(acc[bi][bj][4 * q + e], cn[e] + cnj[bj], kp);
              const int g = ((bi * 4 + q) * 4 + e) * 2 + bj;
              if (g < 32) mlo |= f ? 1u << g : 0u;
              else mhi |= f ? 1u << (g - 32) : 0u;
            }
          }
        }
      }
      const unsigned cnt = (unsigned)(__popc(mlo) + __popc(mhi));
      unsigned pre = cnt;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const unsigned v = __shfl_up(pre, o, 64);
        if (lane >= o) pre += v;
      }
      const unsigned total = __shfl(pre, 63, 64);
      unsigned long long base = 0;
      if (lane == 0 && total) base = atomicAdd(fix_count + seg, (unsigned long long)total);
      base = __shfl(base, 0, 64) + (pre - cnt);
      while (mlo | mhi) {
        const int g = mlo ? __ffs(mlo) - 1 : 32 + __ffs(mhi) - 1;
        if (g < 32) mlo &= mlo - 1u;
        else mhi &= mhi - 1u;
        const int bj = g & 1, e = (g >> 1) & 3, q = (g >> 3) & 3, bi = g >> 5;
        const int64_t gi = row0 + wm * 64 + bi * 32 + 8 * q + 4 * h + e;
        const int64_t gj = col0 + wn * 64 + bj * 32 + l32;
        if (base < (unsigned long long)seg_cap)
          fix_list[(int64_t)seg * seg_cap + (int64_t)base] = make_int2((int)gi, (int)gj);
        ++base;
      }
    }

    // stores of tile (I, J) straight from the MFMA layout (see gemm_kappa_kernel),
    // rows 0-31 of each wavefront's block (bi = 0), then rows 32-63
    char* const Kc = (char*)(Kr + col0);
    const bool full = row0 + kTile <= n && col0 + kTile <= n;
    auto store_rows = [&](int bi) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int iu = bi * 32 + 8 * (r >> 2) + (r & 3);
        char* const rowp = Kc + (size_t)iu * (size_t)S * 4u;
        const float v0 = acc[bi][0][r], v1 = acc[bi][1][r];
        if (full) {
          __builtin_nontemporal_store(v0, (float*)(rowp + lane_b));
          __builtin_nontemporal_store(v1, (float*)(rowp + lane_b + 128u));
          continue;
        }
        if (row0 + wm * 64 + 4 * h + iu >= n) continue;
        const int64_t j0 = col0 + wn * 64 + l32, j1 = j0 + 32;
        if (j0 < ld) __builtin_nontemporal_store(j0 < n ? v0 : 0.f, (float*)(rowp + lane_b));
        if (j1 < ld) __builtin_nontemporal_store(j1 < n ? v1 : 0.f, (float*)(rowp + lane_b + 128u));
      }
    };
    // Packed storage: the next tile's first column block is requested between
    // the two halves of this tile's stores, in registers the products no
    // longer need, so the next tile's first pass of products overlaps the
    // second half of the stores.  (Full storage needs the whole tile for its
    // mirror below, and fetches after it.)
    store_rows(0);
    __builtin_amdgcn_sched_barrier(0);
    if (PACKED && J + 1 < jt1) fetch(J + 1, 0);
    __builtin_amdgcn_sched_barrier(0);
    store_rows(1);
    __builtin_amdgcn_sched_barrier(0);
    if (PACKED && J + 1 < jt1) fetch(J + 1, 1);
    if (!PACKED && J != I) {  // tile (J, I) of full storage: rows j, columns i
#pragma unroll
      for (int bj = 0; bj < 2; ++bj) {
#pragma unroll
        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
          for (int r = 0; r < 16; ++r) Tw[l32 * 65 + bi * 32 + 8 * (r >> 2) + 4 * h + (r & 3)] = acc[bi][bj][r];
        // the wavefront's own LDS tile: its writes complete before its reads
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        const int64_t gj = row0 + wm * 64 + lane;  // I < J, so gj < n
        const int64_t gi0 = col0 + wn * 64 + bj * 32;
        const int nrows = (int)min<int64_t>(32, n - gi0);
        float* dst = K + gi0 * ld + gj;
        if (nrows >= 32) {
#pragma unroll
          for (int rr = 0; rr < 32; ++rr) __builtin_nontemporal_store(Tw[rr * 65 + lane], dst + rr * ld);
        } else {
          for (int rr = 0; rr < nrows; ++rr) __builtin_nontemporal_store(Tw[rr * 65 + lane], dst + rr * ld);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      }
    }
    if (!PACKED && J + 1 < jt1) {
      fetch(J + 1, 0);
      fetch(J + 1, 1);
    }
  }
}

hipError_t launch_gemm_kappa(const float* Xp, const float* nrm, const unsigned* maxnrm_bits,
                             int64_t n, int d_pad, int64_t ld, bool packed, bool f16, const float* kw,
                             const KappaParams& kp, void* K, float* diagK, int2* fix_list,
                             unsigned long long* fix_count, long long seg_cap, const float* bmax, hipStream_t s) {
  if (ld >= kMaxKStride) return hipErrorInvalidValue;
  const int64_t nt = (n + kTile - 1) / kTile;
  if (!f16 && d_pad <= kRegMaxDpad) {
    if (d_pad % 8 || (kp.kind == GAUSS && !bmax)) return hipErrorInvalidValue;
    const int ns = build_sweep_segments(n);
    int64_t items = 0;
    for (int q = 0; q < ns; ++q) items += sweep_seg_begin(q + 1, (int)nt, ns);
    const dim3 sgrid((unsigned)items), sblock(256);
#define KKM_SWEEP(KIND, HP)                                                                                  \
  do {                                                                                                       \
    if (packed)                                                                                              \
      hipLaunchKernelGGL((gemm_kappa_sweep_kernel<KIND, HP, true>), sgrid, sblock, 0, s, Xp, nrm, maxnrm_bits, \
                         n, ld, (int)nt, ns, kp, (float*)K, diagK, fix_list, fix_count, seg_cap, bmax);        \
    else                                                                                                     \
      hipLaunchKernelGGL((gemm_kappa_sweep_kernel<KIND, HP, false>), sgrid, sblock, 0, s, Xp, nrm,             \
                         maxnrm_bits, n, ld, (int)nt, ns, kp, (float*)K, diagK, fix_list, fix_count, seg_cap,  \
                         bmax);                                                                              \
  } while (0)
#define KKM_SWEEP_HP(KIND)                     \
  switch (d_pad / 2) {                         \
    case 4: KKM_SWEEP(KIND, 4); break;         \
    case 8: KKM_SWEEP(KIND, 8); break;         \
    case 12: KKM_SWEEP(KIND, 12); break;       \
    case 16: KKM_SWEEP(KIND, 16); break;       \
    case 20: KKM_SWEEP(KIND, 20); break;       \
    case 24: KKM_SWEEP(KIND, 24); break;       \
    case 28: KKM_SWEEP(KIND, 28); break;       \
    default: KKM_SWEEP(KIND, 32); break;       \
  }
    switch (kp.kind) {
      case LINEAR: KKM_SWEEP_HP(LINEAR); break;
      case POLY: KKM_SWEEP_HP(POLY); break;
      default: KKM_SWEEP_HP(GAUSS); break;
    }
#undef KKM_SWEEP_HP
#undef KKM_SWEEP
    return hipGetLastError();
  }
  const int64_t T = nt * (nt + 1) / 2;
  dim3 grid((unsigned)T), block(256);
#define KKM_GEMM_LAUNCH(KIND, TY)                                                                        \
  hipLaunchKernelGGL((gemm_kappa_kernel<KIND, TY, false>), grid, block, 0, s, Xp, nrm, maxnrm_bits, n,     \
                     d_pad, ld, packed, nt, T, (int64_t)0, n, (int64_t)0, n, kp, (TY*)K, kw, diagK, fix_list, \
                     fix_count, seg_cap)
  switch (kp.kind) {
    case LINEAR:
      if (f16) KKM_GEMM_LAUNCH(LINEAR, half_t);
      else KKM_GEMM_LAUNCH(LINEAR, float);
      break;
    case POLY:
      if (f16) KKM_GEMM_LAUNCH(POLY, half_t);
      else KKM_GEMM_LAUNCH(POLY, float);
      break;
    default:
      if (f16) KKM_GEMM_LAUNCH(GAUSS, half_t);
      else KKM_GEMM_LAUNCH(GAUSS, float);
      break;
  }
#undef KKM_GEMM_LAUNCH
  return hipGetLastError();
}

hipError_t launch_gemm_kappa_panel(const float* Xp, const float* nrm, const unsigned* maxnrm_bits,
                                   int64_t n, int d_pad, int64_t r0, int64_t r1, int64_t c0, int64_t c1,
                                   int64_t ld, const KappaParams& kp, float* K, float* diagK, int2* fix_list,
                                   unsigned long long* fix_count, long long seg_cap, hipStream_t s) {
  if (r0 % kTile || r1 <= r0 || r1 > n || c0 % kTile || c1 <= c0 || c1 > n || ld % kTile || ld < c1 - c0 ||
      ld >= kMaxKStride)
    return hipErrorInvalidValue;
  const int64_t nrow = (r1 - r0 + kTile - 1) / kTile, ncol = ld / kTile;
  const int64_t T = nrow * ncol;
  dim3 grid((unsigned)T), block(256);
#define KKM_PANEL_LAUNCH(KIND)                                                                           \
  hipLaunchKernelGGL((gemm_kappa_kernel<KIND, float, true>), grid, block, 0, s, Xp, nrm, maxnrm_bits, n,   \
                     d_pad, ld, false, ncol, T, r0, r1, c0, c1, kp, K, (const float*)nullptr, diagK,       \
                     fix_list, fix_count, seg_cap)
  switch (kp.kind) {
    case LINEAR: KKM_PANEL_LAUNCH(LINEAR); break;
    case POLY: KKM_PANEL_LAUNCH(POLY); break;
    default: KKM_PANEL_LAUNCH(GAUSS); break;
  }
#undef KKM_PANEL_LAUNCH
  return hipGetLastError();
}

// ---- Gaussian fix-up: |x_i - x_j|^2 summed from the coordinate differences.
//
// Both passes below evaluate a recomputed entry with the same routine: a group
// of 16 lanes, lane gl summing the float4 chunks gl, gl + 16, ... in order,
// then a fixed shuffle tree over the group.  So an entry recomputed twice gets
// the same bits, and its mirror (written by the same lane) equals it.
__device__ inline float sqdist_group16(const float* __restrict__ Xp, int64_t i, int64_t j, int d_pad, int gl) {
  const float4* xi = (const float4*)(Xp + i * d_pad);
  const float4* xj = (const float4*)(Xp + j * d_pad);
  const int nq = d_pad >> 2;
  float s = 0.f;
  for (int cc = gl; cc < nq; cc += 16) {
    const float4 a = xi[cc], b = xj[cc];
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
  return s;
}

// Store a recomputed entry (i, j) and, in the square layouts, its mirror.  A
// block (c1 > 0: rows [r0, r1) and columns [c0, c1) stored at (i - r0, j - c0))
// stores each of its entries once; the square layouts get pairs with i < j.
template <typename T>
__device__ inline void store_fixed(T* __restrict__ K, int64_t i, int64_t j, float s, int64_t ld, bool packed,
                                   int64_t r0, int64_t c0, bool panel, const KappaParams& kp) {
  const T v = (T)__builtin_amdgcn_exp2f(kp.neg_g_log2e * s);
  if (panel) {
    K[(i - r0) * ld + (j - c0)] = v;
  } else if (packed) {
    K[packed_row(i, ld) + j] = v;
    if (i / kTile == j / kTile) K[packed_row(j, ld) + i] = v;
  } else {
    K[i * ld + j] = v;
    K[j * ld + i] = v;
  }
}

__device__ inline bool fix_list_overflowed(const unsigned long long* __restrict__ counts, long long seg_cap) {
  __shared__ int overflow;
  if (threadIdx.x == 0) overflow = 0;
  __syncthreads();
  for (int q = threadIdx.x; q < kFixSegs; q += blockDim.x)
    if (counts[q] > (unsigned long long)seg_cap) overflow = 1;
  __syncthreads();
  return overflow != 0;
}

// Pass 1: the listed pairs.  Workgroups b, b + kFixSegs, ... share list
// segment b % kFixSegs; a group of 16 lanes per pair.
template <typename T>
__global__ __launch_bounds__(256) void gauss_fixup_kernel(const float* __restrict__ Xp, int d_pad, int64_t ld,
                                                          bool packed, int64_t r0, int64_t c0, bool panel,
                                                          KappaParams kp, const int2* __restrict__ list,
                                                          const unsigned long long* __restrict__ counts,
                                                          long long seg_cap, T* __restrict__ K) {
  const int seg = (int)(blockIdx.x % kFixSegs), part = (int)(blockIdx.x / kFixSegs);
  const int parts = (int)(gridDim.x / kFixSegs);
  const unsigned long long c = counts[seg];
  const long long count = c < (unsigned long long)seg_cap ? (long long)c : seg_cap;
  const int2* seg_list = list + (int64_t)seg * seg_cap;
  const int g = threadIdx.x >> 4, gl = threadIdx.x & 15;
  for (long long p = (long long)part * 16 + g; p < count; p += (long long)parts * 16) {
    const int2 ij = seg_list[p];
    const float s = sqdist_group16(Xp, ij.x, ij.y, d_pad, gl);
    if (gl == 0) store_fixed(K, ij.x, ij.y, s, ld, packed, r0, c0, panel, kp);
  }
}

// Pass 2, launched after pass 1 and only doing work when some list segment
// received more entries than it holds: every entry of the upper triangle (of
// the block) is re-tested from the stored K with the epilogue's estimate.
// Each wavefront tests 64 entries at once and recomputes the flagged ones
// four at a time, one 16-lane group each.  An entry pass 1 already fixed may
// be flagged again; it is recomputed to the same value.
template <typename T>
__global__ __launch_bounds__(256) void gauss_refix_kernel(const float* __restrict__ Xp,
                                                          const float* __restrict__ nrm, int64_t n, int d_pad,
                                                          int64_t ld, bool packed, int64_t r0, int64_t r1,
                                                          int64_t c0, int64_t c1, KappaParams kp,
                                                          const unsigned long long* __restrict__ counts,
                                                          long long seg_cap, T* __restrict__ K) {
  if (!fix_list_overflowed(counts, seg_cap)) return;
  const bool panel = c1 > 0;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g = lane >> 4, gl = lane & 15;
  const int64_t ilo = panel ? r0 : 0, ihi = panel ? r1 : n;
  for (int64_t i = ilo + blockIdx.x; i < ihi; i += gridDim.x) {  // uniform over the workgroup
    const float ni = nrm[i];
    const int64_t jlo = panel ? c0 : i + 1, jhi = panel ? c1 : n;
    const int64_t ri = panel ? (i - r0) * ld - c0 : (packed ? packed_row(i, ld) : i * ld);
    for (int64_t jb = jlo + wave * 64; jb < jhi; jb += 256) {  // uniform over the wavefront
      const int64_t j = jb + lane;
      bool need = false;
      if (j < jhi && j != i) need = gauss_needs_fix((float)K[ri + j], ni, nrm[j], kp);
      uint64_t m = __ballot(need);
      while (m) {
        // group g takes the g-th lowest flagged lane of this round
        uint64_t mm = m;
        int src = -1;
        for (int q = 0; q <= g; ++q) {
          if (!mm) {
            src = -1;
            break;
          }
          src = __ffsll((unsigned long long)mm) - 1;
          mm &= mm - 1;
        }
        const int64_t jj = jb + (src < 0 ? 0 : src);
        const float s = sqdist_group16(Xp, i, src < 0 ? i : jj, d_pad, gl);
        if (src >= 0 && gl == 0) store_fixed(K, i, jj, s, ld, packed, r0, c0, panel, kp);
        for (int q = 0; q < 4 && m; ++q) m &= m - 1;
      }
    }
  }
}

hipError_t launch_gauss_fixup(const float* Xp, const float* nrm, int64_t n, int d_pad, int64_t ld,
                              bool packed, bool f16, const KappaParams& kp, const int2* fix_list,
                              const unsigned long long* fix_count, long long seg_cap, void* K,
                              hipStream_t s, int64_t r0, int64_t r1, int64_t c0, int64_t c1) {
  const bool panel = c1 > 0;
  const dim3 grid(16 * kFixSegs), block(256);
  if (f16) {
    hipLaunchKernelGGL(gauss_fixup_kernel<half_t>, grid, block, 0, s, Xp, d_pad, ld, packed, r0, c0, panel, kp,
                       fix_list, fix_count, seg_cap, (half_t*)K);
    hipLaunchKernelGGL(gauss_refix_kernel<half_t>, grid, block, 0, s, Xp, nrm, n, d_pad, ld, packed, r0, r1, c0,
                       c1, kp, fix_count, seg_cap, (half_t*)K);
  } else {
    hipLaunchKernelGGL(gauss_fixup_kernel<float>, grid, block, 0, s, Xp, d_pad, ld, packed, r0, c0, panel, kp,
                       fix_list, fix_count, seg_cap, (float*)K);
    hipLaunchKernelGGL(gauss_refix_kernel<float>, grid, block, 0, s, Xp, nrm, n, d_pad, ld, packed, r0, r1, c0,
                       c1, kp, fix_count, seg_cap, (float*)K);
  }
  return hipGetLastError();
}

}  // namespace kkm
