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
// which runs on the matrix cores with 16 labels per block, exact in its
// products (each is 0 or the operand itself):
//  - binary16 K: v_mfma_f32_16x16x32_f16, 32 columns per instruction;
//  - fp32 K: each entry v of row r, divided by p_r, a power of two at or
//    above a bound of |K(r, .)| (1 for the Gaussian, whose entries lie in
//    [0, 1]; the Cauchy-Schwarz row bound otherwise), as the sum of two
//    binary16 values, hi = its rounding and lo = the rest rounded, on
//    v_mfma_f32_16x16x32_f16: 32 columns per two instructions.  hi + lo is
//    within 2^-22 |v / p_r| of v / p_r, or 2^-25 absolute below binary16's
//    normal range; the row's sums are multiplied by p_r again (exact) and
//    stay fp32.  On the fp32 matrix instruction (4 columns each) the column
//    side outweighed the HBM time above 32 labels; split, it stays below it
//    up to 64.
// The k slots of an instruction are summed over, so any order of the
// columns over them is right as long as the one-hot operand and the entries
// take the same one: each lane puts the 4 columns of its slot in column
// group g, then the 4 of group g + 1.
//
// Workgroup (chunk q, segment sg): NW wavefronts (4 or 8), one 16-row group
// each, over the column tiles of segment sg (BSEG tiles) that the chunk's
// rows store.
// Per step (one tile of fp32 K, two of binary16) a wavefront
//  - streams its 16 rows with 16-byte loads, two rows of 512 contiguous
//    bytes per instruction, one step ahead in a single register buffer (a
//    second one, with the rows' offsets moved to LDS to make room, measured
//    no faster on the largest problems and slower on smaller ones);
//  - adds the rows in registers (row side), combines the wavefronts in LDS
//    and writes the chunk's partial P[q] for the step's columns;
//  - stages each block in LDS and reads it back in the MFMA operand layout
//    (lane = row, k slot = column) for the column side.  The next step's
//    loads are issued once the step's last block is staged, so they are in
//    flight during its multiply.
// The scatter writes, once per update, the chunks' members in chunk-major
// order and each column tile's one-hot bits, so a workgroup's prologue is a
// single round trip of independent loads.  With one label block the
// segment's bits are staged in LDS; with more, each tile's are loaded with
// its entries (the LDS holds the whole staged block instead).  The
// column-side sums of a row stay in the accumulators for the whole segment
// and go to the workgroup's contiguous k x R block of Ecp (label-major, rows
// at their chunk positions); ecol_sum_kernel adds the segments into Ecol at
// each row's point index, and spmm_reduce_sym_kernel adds them into E^T.
// Fixed orders throughout, so the result is bitwise reproducible.
#include "kkm_internal.h"

#include <algorithm>
#include <climits>
#include <type_traits>

namespace kkm {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));

namespace {

// The smallest power of two at or above w, for w up to 2^126 (larger w,
// infinities and NaN give 2^126; w <= 0 does not occur: the bounds are
// positive).
__device__ inline float pow2_at_least(float w) {
  w = fminf(w, 0x1p126f);
  return __uint_as_float((__float_as_uint(w) + 0x007fffffu) & 0x7f800000u);
}

// 102-128 VGPRs and 25-39 KB (NW = 4) or 50-78 KB (NW = 8) of LDS per
// workgroup: 16 wavefronts per CU.  Six wavefronts per SIMD (80 VGPRs,
// spilling) measured slower.
// KT: float, or binary16 with row r's entries divided by kw[r] (kw null: 1),
// widened and scaled in the row side; the column side scales the row's sums
// once at the end.
template <int NB, int NW, int BSEG, typename KT>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(4))) void spmm_sym_kernel(
    const KT* __restrict__ Kp, IterBufs b) {
  constexpr bool kHalf = sizeof(KT) == 2;
  using BufT = typename std::conditional<kHalf, h8, f4>::type;  // a lane's 16 bytes of a row
  constexpr int R = 16 * NW, NT = 64 * NW;
  // binary16: a step takes two tiles, read 8 entries (16 bytes) per lane
  // like fp32's 4, so an instruction reads two rows of 512 contiguous bytes;
  // its rows come from the LDS row table
  constexpr bool kPair = kHalf;
  constexpr bool kFull = NB == 1 && !kPair;
  constexpr int kTps = kPair ? 2 : 1;           // tiles per step
  constexpr int kStepCols = kTps * kTile;       // columns of P per step
  constexpr int kLc = 16 / (int)sizeof(KT);     // entries per lane and row
  // With more than one label block each tile's one-hot bits (NB x 256 bytes)
  // are read from global memory with its entries instead of a whole
  // segment's being staged in LDS: the LDS then holds the whole staged block,
  // so the next tile's loads are issued as soon as it is staged, and
  // segments can be long.
  constexpr bool kTileMask = NB > 1;
  constexpr int kCh = kHalf ? 16 : 32;                   // 16-byte chunks per staged row
  constexpr int kMw = BSEG * NB * 64;                    // one-hot words of a segment
  constexpr int kMpt = (kMw + NT - 1) / NT;              // ... per thread
  const int nseg = b.nseg;
  const int q = (int)(blockIdx.x / (unsigned)nseg), sg = (int)(blockIdx.x % (unsigned)nseg);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int li = lane & 15, lk = lane >> 4;   // MFMA layout: row li, k slot lk
  const int h = lane >> 5, c32 = lane & 31;   // load layout: row 2g + h, columns 4*c32 .. +3
  const int64_t ld = b.ld;
  const int Js = sg * BSEG, Je = min(b.nt, Js + BSEG);

  // Everything the workgroup needs is read in one round trip: the chunk's
  // rows by point index from the scatter's chunk-major table (-1 past the
  // chunk's end and at the start of an unused chunk), and with one label
  // block the segment's one-hot bits (bit 4g+e of [tile][nb][lk][li]: column
  // 16g + 4lk + e of the tile has label 16nb + li).
  const int* cr = b.crow + (int64_t)q * R;
  const int i0 = cr[0];
  const int um = w * 16 + li;  // this lane's row in the MFMA layout
  const int im = cr[um];
  int iu[8];
  if (kFull) {
#pragma unroll
    for (int g = 0; g < 8; ++g) iu[g] = cr[w * 16 + 2 * g + h];
  }
  const int64_t mbase = (int64_t)Js * NB * 64, mlast = (int64_t)b.nt * NB * 64 - 1;
  unsigned mv[kMpt];
#pragma unroll
  for (int m = 0; m < kMpt; ++m) mv[m] = kTileMask ? 0u : b.mskg[min(mbase + tid + m * NT, mlast)];
  // Rows are in increasing index order within a chunk, so the first row has
  // the smallest tile; a segment left of it holds nothing of this chunk.
  if (i0 < 0 || i0 / kTile >= Je) return;

  __shared__ int rtile[kFull ? 1 : R];
  __shared__ int64_t roff[kFull ? 1 : R];
  __shared__ float rwl[kHalf ? R : 1];           // row scales (binary16)
  __shared__ unsigned mskl[kTileMask ? 1 : BSEG][NB][4][16];  // one-hot bits: [tile][label block][k slot][label]
  __shared__ f4 tile[NW][16 * kCh];              // per wavefront: 16 rows x kCh chunks of 16 B
  __shared__ f4 red[2][NW][kStepCols / 4];       // row-side sums of the wavefronts
  __shared__ h4 onehot[16];                      // the 4 bits of a nibble as binary16 0 / 1
  __shared__ float rsc[kHalf ? 1 : R];           // fp32 K: the rows' column-side scales

  const int I0 = i0 / kTile;
  const int J_lo = max(Js, I0), J_hi = Je;
  const int rt_m = im >= 0 ? im / kTile : INT_MAX;
  // first and last diagonal tile among the wavefront's 16 rows (rows increase
  // with their position in the chunk; lane 0 holds the first)
  const int rt_first = __shfl(rt_m, 0, 64);
  int rt_last = im >= 0 ? rt_m : -1;
#pragma unroll
  for (int off = 1; off < 16; off <<= 1) rt_last = max(rt_last, __shfl_xor(rt_last, off, 16));

  // This lane's 8 rows (2g + h of its wavefront's group).  Rows not stored
  // in tile J (their diagonal tile is further right), rows past the chunk and
  // tiles past the segment read the zero page instead, so the loads need no
  // branch.  With one label block the rows' packed bases (at this lane's 4
  // columns of tile 0) and diagonal tiles are held in registers, so issuing
  // a tile's loads needs no LDS round trip; with more label blocks the
  // registers go to the accumulators and the rows are read from LDS.
  const KT* rbase[8];
  int rt[8];
  float rwt[8];
  if (kFull) {
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      rt[g] = iu[g] >= 0 ? iu[g] / kTile : INT_MAX;
      rbase[g] = Kp + packed_row(iu[g] >= 0 ? iu[g] : 0, ld) + 4 * c32;
      if (kHalf) rwt[g] = (iu[g] >= 0 && b.kw) ? b.kw[iu[g]] : 1.f;
    }
  } else if (tid < R) {
    const int iv = cr[tid];
    rtile[tid] = iv >= 0 ? iv / kTile : INT_MAX;
    roff[tid] = iv >= 0 ? packed_row(iv, ld) : 0;
    if (kHalf) rwl[tid] = (iv >= 0 && b.kw) ? b.kw[iv] : 1.f;
  }
  const KT* zp = (const KT*)b.zero + kLc * c32;
  // the step's rows at lane column kLc * c32 from tile J (binary16: lanes
  // c32 < 16 in tile J, the others in J + 1), and with more label blocks
  // the tiles' one-hot bits
  auto load = [&](BufT(&buf)[8], unsigned(&mk)[kTps][NB], int J) {
    if constexpr (kTileMask) {
#pragma unroll
      for (int t = 0; t < kTps; ++t)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          mk[t][nb] = b.mskg[min(((int64_t)(J + t) * NB + nb) * 64 + lk * 16 + li, mlast)];
    }
    const int jt = kPair ? J + (c32 >> 4) : J;  // this lane's tile
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      const int u = w * 16 + 2 * g + h;
      const bool on = (kFull ? rt[g] : rtile[u]) <= jt && jt < J_hi;
      const KT* rp = kFull ? rbase[g] + (int64_t)J * kTile : Kp + roff[u] + (int64_t)J * kTile + kLc * c32;
      buf[g] = __builtin_nontemporal_load((const BufT*)(on ? rp : zp));
    }
  };

  BufT bb[8];
  unsigned mk[kTps][NB];
  if (kFull) load(bb, mk, J_lo);  // in flight while the one-hot bits go to LDS
  // fp32 K: row u of the chunk is scaled by rsc[u], a power of two, for the
  // column side (exact both ways; read per tile, so it holds no register)
  if (!kHalf && tid < R) {
    const int iv = cr[tid];
    rsc[tid] = iv >= 0 && b.kw ? 1.f / pow2_at_least(b.kw[iv]) : 1.f;
  }
  if (tid < 16)
    onehot[tid] = h4{(_Float16)(tid & 1), (_Float16)((tid >> 1) & 1), (_Float16)((tid >> 2) & 1),
                     (_Float16)((tid >> 3) & 1)};
  if constexpr (!kTileMask) {
#pragma unroll
    for (int m = 0; m < kMpt; ++m)
      if (tid + m * NT < kMw) (&mskl[0][0][0][0])[tid + m * NT] = mv[m];
  }
  __syncthreads();
  if (!kFull) load(bb, mk, J_lo);

  f4 D[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) D[nb] = f4{0.f, 0.f, 0.f, 0.f};
  f4* tw = tile[w];

  // row side: this lane's columns over its 8 rows, then the other
  // half-wave's 8 (binary16: widened and scaled by the row); rs[t] holds
  // columns kLc * c32 + 4t .. +3 of the step
  auto rowsum = [&](const BufT(&raw)[8], f4(&rs)[kTps]) {
#pragma unroll
    for (int g = 0; g < 8; ++g) {
#pragma unroll
      for (int t = 0; t < kTps; ++t) {
        f4 v;
        if constexpr (kHalf) {
          const h4 x = t == 0 ? __builtin_shufflevector(raw[g], raw[g], 0, 1, 2, 3)
                              : __builtin_shufflevector(raw[g], raw[g], 4, 5, 6, 7);
          v = __builtin_convertvector(x, f4) * (kFull ? rwt[g] : rwl[w * 16 + 2 * g + h]);
        } else {
          v = raw[g];
        }
        rs[t] = g == 0 ? v : rs[t] + v;
      }
    }
#pragma unroll
    for (int t = 0; t < kTps; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e) rs[t][e] += __shfl_xor(rs[t][e], 32, 64);
  };
  // tile J's one-hot bits (J inside the segment)
  auto bits = [&](unsigned(&msk)[NB], const unsigned(&mkr)[NB], int J) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) msk[nb] = kTileMask ? mkr[nb] : mskl[kTileMask ? 0 : J - Js][nb][lk][li];
  };
  // Column side of tile J for the group: entries right of each row's own
  // diagonal tile.  diag: some row of the group sits in tile J; dz: this
  // lane's row sits in tile J or right of it (its entries there are row side
  // only); any: the group has column-side entries in tile J (wavefront-uniform).
  auto diag_at = [&](int J) { return rt_first <= J && J <= rt_last; };
  auto any_at = [&](int J) { return rt_first < J || diag_at(J); };
  // The row side across the wavefronts -> P[q]: each wavefront's sums to
  // its slot, then the step's columns from tile J (ncols of them are
  // written; the rest belong to the next segment).
  auto put_rows = [&](const f4(&rs)[kTps], int par) {
    if (h == 0)
#pragma unroll
      for (int t = 0; t < kTps; ++t) red[par][w][kTps * c32 + t] = rs[t];
  };
  auto combine = [&](int J, int par, int ncols) {
    __syncthreads();
    if (tid < ncols) {
      const float* rr = (const float*)red[par];
      float t = rr[tid];
#pragma unroll
      for (int ww = 1; ww < NW; ++ww) t += rr[ww * kStepCols + tid];
      b.P[(int64_t)q * ld + (int64_t)J * kTile + tid] = t;
    }
  };

  // fp32 K, one tile per step.  The block is staged in LDS (chunk index xor
  // row keeps both the row-wise writes and the MFMA-layout reads
  // conflict-free) and read back in the MFMA operand layout.  The next
  // tile's loads are issued as soon as the whole block is staged, so they
  // are in flight while it is multiplied.  The row's entries (scaled into
  // [-1, 1]) go in as a sum of two binary16 values (hi, and the rest
  // rounded).  Column groups g and g + 1 go to one v_mfma_f32_16x16x32_f16
  // (k slots 0-3 and 4-7 of each lane; the one-hot operand takes the same
  // order): 32 columns per instruction and label block, exact 0/1 products,
  // fp32 sums.
  auto step = [&](auto& raw, auto& mkr, int J, int par) {  // (generic: instantiated for fp32 only)
    f4 rs[kTps];
    rowsum(raw, rs);
    unsigned msk[NB];
    bits(msk, mkr[0], J);
    const bool diag = diag_at(J), dz = rt_m >= J;
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      const int r = 2 * g + h;
      tw[r * 32 + (c32 ^ r)] = raw[g];
    }
    __builtin_amdgcn_sched_barrier(0);
    load(raw, mkr, J + 1);
    __builtin_amdgcn_sched_barrier(0);
    if (any_at(J)) {
      const float ips = rsc[um];
#pragma unroll
      for (int g = 0; g < 8; g += 2) {
        f4 v0 = tw[li * 32 + ((4 * g + lk) ^ li)];      // row li, columns 16g + 4lk .. +3
        f4 v1 = tw[li * 32 + ((4 * g + 4 + lk) ^ li)];  // ... and 16(g+1) + 4lk .. +3
        if (diag && dz) v0 = v1 = f4{0.f, 0.f, 0.f, 0.f};
        v0 *= ips;
        v1 *= ips;
        const h4 h0 = __builtin_convertvector(v0, h4), h1 = __builtin_convertvector(v1, h4);
        const h4 l0 = __builtin_convertvector(v0 - __builtin_convertvector(h0, f4), h4);
        const h4 l1 = __builtin_convertvector(v1 - __builtin_convertvector(h1, f4), h4);
        const h8 hi = __builtin_shufflevector(h0, h1, 0, 1, 2, 3, 4, 5, 6, 7);
        const h8 lo = __builtin_shufflevector(l0, l1, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const h8 a = __builtin_shufflevector(onehot[(msk[nb] >> (4 * g)) & 15u],
                                               onehot[(msk[nb] >> (4 * g + 4)) & 15u], 0, 1, 2, 3, 4, 5, 6, 7);
          D[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, hi, D[nb], 0, 0, 0);
          D[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, lo, D[nb], 0, 0, 0);
        }
      }
    }
    put_rows(rs, par);
    combine(J, par, kTile);
  };

  // binary16 K: a step's two blocks go through the wavefront's staging area
  // in turn (4 KB; 8-byte chunk c of row r at c ^ 2r, conflict-free for the
  // row-wise writes and for the operand reads, which LDS serves 32 lanes at a
  // time; a wavefront's LDS accesses are carried out in order, so the second
  // block's writes follow the first block's reads), and the column side runs
  // on v_mfma_f32_16x16x32_f16: 32 columns per instruction and label block,
  // the one-hot operand from a table of the 16 nibbles; the products are
  // exact and the sums fp32, and the row's scale is applied at the end.  The
  // next step's loads are issued once the second block is staged, and the
  // row sums go to LDS as soon as they are formed (the previous step's
  // barrier ended the reads of their slot), so they hold no registers.
  auto stage16 = [&](const BufT(&raw)[8], int t) {  // the block of tile J + t
    if constexpr (kPair) {
      if ((c32 >> 4) != t) return;
      h8* th = (h8*)tw;
      const int cc = c32 & 15;  // chunks 2cc, 2cc + 1 of the block's row
#pragma unroll
      for (int g = 0; g < 8; ++g) {
        const int r = 2 * g + h;
        th[r * 16 + (cc ^ r)] = raw[g];
      }
    }
  };
  auto mma16 = [&](int J, const unsigned(&msk)[NB]) {
    const bool diag = diag_at(J), dz = rt_m >= J;
    const h4* th = (const h4*)tw;
#pragma unroll
    for (int g = 0; g < 8; g += 2) {  // column groups g and g + 1 per instruction
      const h4 v0 = th[li * 32 + ((4 * g + lk) ^ (2 * li))];  // row li, columns 16g + 4lk .. +3
      const h4 v1 = th[li * 32 + ((4 * g + 4 + lk) ^ (2 * li))];
      h8 v = __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
      if (diag && dz) v = h8{0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const h8 a = __builtin_shufflevector(onehot[(msk[nb] >> (4 * g)) & 15u],
                                             onehot[(msk[nb] >> (4 * g + 4)) & 15u], 0, 1, 2, 3, 4, 5, 6, 7);
        D[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, v, D[nb], 0, 0, 0);
      }
    }
  };
  auto step2 = [&](auto J, int par) {  // (generic: instantiated for binary16 only)
    const bool two = J + 1 < J_hi;    // tile J + 1 is in the segment
    {
      f4 rs[kTps];
      rowsum(bb, rs);
      put_rows(rs, par);
    }
    unsigned msk[NB];
    bits(msk, mk[0], J);
    stage16(bb, 0);
    if (any_at(J)) mma16(J, msk);
    bits(msk, mk[kTps - 1], two ? J + 1 : J);
    stage16(bb, kTps - 1);
    __builtin_amdgcn_sched_barrier(0);
    load(bb, mk, J + 2);
    __builtin_amdgcn_sched_barrier(0);
    if (two && any_at(J + 1)) mma16(J + 1, msk);
    combine(J, par, two ? 2 * kTile : kTile);
  };

  if constexpr (kPair) {
    for (int J = J_lo; J < J_hi; J += 2) step2(J, ((J - J_lo) >> 1) & 1);
  } else {
    for (int J = J_lo; J < J_hi; ++J) step(bb, mk, J, (J - J_lo) & 1);
  }

  // D[nb][r]: label 16nb + 4lk + r of row um, at its chunk-major position
  // (binary16 on the matrix path: sums of the stored values, times the row's scale)
  if constexpr (kHalf) {
    const float wm = (im >= 0 && b.kw) ? b.kw[im] : 1.f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) D[nb] *= wm;
  }
  if constexpr (!kHalf) {
    const float ps = 1.f / rsc[um];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) D[nb] *= ps;
  }
  // the workgroup's k x R block of Ecp is contiguous
  float* ep = b.Ecp + ((int64_t)sg * b.qmax + q) * b.k * R + um;
  if (im >= 0)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int lab = 16 * nb + 4 * lk + r;
        if (lab < b.k) ep[lab * R] = D[nb][r];
      }
}

// Ecol[j][i] = the column-side sums of point i (member u of chunk q) over
// the segments that hold its row's stored columns, in order.  One output per
// thread: (chunk, label, member) over ecol_wgs(b) workgroups per chunk.
__device__ __host__ inline int ecol_wgs(const IterBufs& b) { return (b.k * b.chunk_len + 255) / 256; }
__global__ __launch_bounds__(256) void ecol_sum_kernel(IterBufs b) {
  const int per = ecol_wgs(b), cl = b.chunk_len;
  const int q = (int)(blockIdx.x / (unsigned)per), part = (int)(blockIdx.x % (unsigned)per);
  const int t = part * 256 + (int)threadIdx.x;
  const int j = t / cl, u = t % cl;
  const int* cr = b.crow + (int64_t)q * cl;
  const int i0 = cr[0], row = cr[u];
  if (i0 < 0 || j >= b.k || row < 0) return;
  const int s0 = i0 / kTile / b.bseg, last = b.nseg - 1;
  const int64_t seg_stride = (int64_t)b.qmax * b.k * cl;
  const float* e = b.Ecp + ((int64_t)q * b.k + j) * cl + u;  // = chunk q's block + t
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
    // a chunk's partial starts at its first stored column: entries left of
    // it are stale and are not read
    for (int q = q0; q < q1; q += 8) {  // eight chunks in flight, added in order
      int c0[8];
      f4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) c0[u] = b.chunk_c0[min(q + u, q1 - 1)];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        v[u] = f4{0.f, 0.f, 0.f, 0.f};
        if (q + u < q1 && col >= c0[u]) v[u] = *(const f4*)(b.P + (int64_t)(q + u) * ld + col);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) e += v[u];
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
// (binary16: widened and scaled by the row that stores the entry)
template <typename KT>
__global__ __launch_bounds__(256) void packed_rows_kernel(const KT* __restrict__ Kp, const float* __restrict__ kw,
                                                          int64_t n, int64_t ld, int64_t r0, int64_t r1,
                                                          float* __restrict__ out) {
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (c >= n) return;
  for (int64_t r = r0 + blockIdx.y; r < r1; r += gridDim.y) {
    const int64_t c0 = (r / kTile) * kTile;
    const int64_t sr = c >= c0 ? r : c;  // the row that stores K(r, c)
    const float v = (float)Kp[packed_row(sr, ld) + (c >= c0 ? c : r)];
    out[(r - r0) * n + c] = kw ? v * kw[sr] : v;
  }
}

}  // namespace

hipError_t launch_spmm_sym(const void* Kp, const IterBufs& b, hipStream_t s) {
  const unsigned grid = (unsigned)((int64_t)b.qmax * b.nseg);
  const int nb = b.nlb;
  if (nb != (b.k + 15) / 16) return hipErrorInvalidValue;
#define KKM_SYM_LAUNCH(NB, NW, S)                                                                        \
  do {                                                                                                   \
    if (b.kf16)                                                                                          \
      hipLaunchKernelGGL((spmm_sym_kernel<NB, NW, S, half_t>), dim3(grid), dim3(64 * NW), 0, s,            \
                         (const half_t*)Kp, b);                                                          \
    else                                                                                                 \
      hipLaunchKernelGGL((spmm_sym_kernel<NB, NW, S, float>), dim3(grid), dim3(64 * NW), 0, s,             \
                         (const float*)Kp, b);                                                           \
  } while (0)
  // the segment lengths sym_seg_for sets
  const bool tall = b.chunk_len == 128;
  const int lo = nb == 1 ? 2 : 8, hi = nb == 1 ? 8 : 16;  // short chunks: the two smaller lengths
  const bool ok = tall ? (nb == 1 ? b.bseg == 16 : b.bseg == 32 || b.bseg == 64) : b.bseg == lo || b.bseg == hi;
  if (!ok) return hipErrorInvalidValue;
#define KKM_SYM_CASE(NB, LO, HI)                                         \
  do {                                                                   \
    if (tall && b.bseg == 64) KKM_SYM_LAUNCH(NB, 8, 64);                 \
    else if (tall) KKM_SYM_LAUNCH(NB, 8, 2 * HI);                        \
    else if (b.bseg == LO) KKM_SYM_LAUNCH(NB, 4, LO);                    \
    else KKM_SYM_LAUNCH(NB, 4, HI);                                      \
  } while (0)
  switch (nb) {
    case 1:
      if (tall) KKM_SYM_LAUNCH(1, 8, 16);
      else if (b.bseg == 2) KKM_SYM_LAUNCH(1, 4, 2);
      else KKM_SYM_LAUNCH(1, 4, 8);
      break;
    case 2: KKM_SYM_CASE(2, 8, 16); break;
    case 3: KKM_SYM_CASE(3, 8, 16); break;
    case 4: KKM_SYM_CASE(4, 8, 16); break;
    default: return hipErrorInvalidValue;  // k > kSymMaxK is rejected before launch
  }
#undef KKM_SYM_CASE
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

hipError_t launch_packed_rows(const void* Kp, bool f16, const float* kw, int64_t n, int64_t ld, int64_t r0,
                              int64_t r1, float* out, hipStream_t s) {
  const unsigned gy = (unsigned)std::min<int64_t>(r1 - r0, 65535);
  const dim3 grid((unsigned)((n + 255) / 256), gy);
  if (f16)
    hipLaunchKernelGGL(packed_rows_kernel<half_t>, grid, dim3(256), 0, s, (const half_t*)Kp, kw, n, ld, r0, r1, out);
  else
    hipLaunchKernelGGL(packed_rows_kernel<float>, grid, dim3(256), 0, s, (const float*)Kp, nullptr, n, ld, r0, r1,
                       out);
  return hipGetLastError();
}
}  // namespace kkm
