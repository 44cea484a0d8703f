// Internal declarations shared by the engine's HIP translation units.
// Every kernel here is written for gfx950 (CDNA4: 64-lane wavefronts, fp32
// MFMA, 160 KB LDS per CU, 8 XCDs with private L2s).
#pragma once
#include <hip/hip_runtime.h>
#include <cstddef>
#include <cstdint>

namespace kkm {

// K-build tiling: 128 x 128 output tile per 256-thread workgroup (2 x 2
// wavefronts, each 64 x 64 = 2 x 2 MFMA 32x32 blocks), 16-wide k chunks.
constexpr int kTile = 128;
constexpr int kBK = 16;
// The K build addresses a tile's fp32 stores as a row base plus a 32-bit
// byte offset of at most (127 S + 128) * 4 for the row stride S, so every
// layout keeps S below kMaxKStride floats (a square K that wide would not
// fit in memory; a panel or block is checked when it is built).
constexpr int64_t kMaxKStride = (int64_t)1 << 23;

// One-hot SpMM: a workgroup streams a stripe of kStripe columns of K over a
// chunk of at most kChunk rows that all belong to one cluster (long chunks:
// fewer workgroup prologues and partial sums; 1024 rows measured best).
constexpr int kStripe = 1024;
constexpr int kChunk = 1024;

// Points per workgroup in the label/assign/scatter kernels.
constexpr int kBlk = 256;

// Packed (upper block triangle) SpMM: a workgroup of W wavefronts takes a
// chunk of at most 16 W sorted rows of one cluster (one 16-row MFMA group per
// wavefront) and a segment of S column tiles.  Up to kSymSmallN points W = 4,
// above it W = 8 (taller chunks halve the partial sums).  S by problem size:
//                          k <= 16   k > 16
//   n <= kSymTinyN            2         8
//   n <= kSymSmallN           8        16
//   n <= kSymLargeN          16        32
//   n >  kSymLargeN          16        64
// Small problems need many workgroups to fill the GPU evenly (2000 points,
// k = 8: 18.8 us per SpMM at S = 8, 11.4 at S = 2).  Longer segments spread
// each workgroup's start (row addresses far apart in a K of tens of GB) over
// more tiles, and each workgroup writes k column-side sums per row of its
// chunk for its segment, which the next kernel reads back: with more labels
// these partials and the epilogue weigh more against the tiles streamed.
// SpMM per launch, binary16 column side, k = 64: 200000 points 17.0 / 15.6 /
// 13.6 ms at S = 8 / 16 / 32; 100000 points 3.92 ms at S = 32, 3.79 at 64;
// 60000 points 1.38 ms at S = 32, 2.01 at 64 (too few workgroups: about
// (n/128)^2 / 2S chunk segments against 512 at a time); 20000 points S = 16
// beats 8 and 32.  With one label block S = 16 and 32 measured alike.
// kSymMaxK bounds the one-hot MFMA label blocks (16 labels each) a wavefront
// carries.
constexpr int64_t kSymSmallN = 40000, kSymTinyN = 4096, kSymLargeN = 90000;
inline int sym_chunk_for(int64_t n) { return n <= kSymSmallN ? 64 : 128; }
inline int sym_seg_for(int64_t n, int k) {
  if (n <= kSymTinyN) return k <= 16 ? 2 : 8;
  if (n <= kSymSmallN) return k <= 16 ? 8 : 16;
  if (n <= kSymLargeN) return k <= 16 ? 16 : 32;
  return k <= 16 ? 16 : 64;
}
constexpr int kSymMaxK = 64;
constexpr int kSymRedStripe = 256;  // columns per workgroup of the packed reduction

// Packed layout: row block I (rows I*kTile ..) stores columns I*kTile ..
// ld-1 row-major with stride ld - I*kTile.  packed_row(i) is the offset of
// the (unstored when I > 0) element (i, 0), so that (i, j) for
// j >= kTile*(i/kTile) lives at packed_row(i) + j.
__host__ __device__ inline int64_t packed_row(int64_t i, int64_t ld) {
  const int64_t I = i / kTile, c0 = I * kTile;
  return kTile * (I * ld - (int64_t)kTile * I * (I - 1) / 2) + (i - c0) * (ld - c0) - c0;
}
// Floats held by the packed K of n rows (ld a multiple of kTile): the last
// stored element is (n-1, ld-1).
inline int64_t packed_floats(int64_t n, int64_t ld) { return packed_row(n - 1, ld) + ld; }

// The Gaussian fix-up list is split into kFixSegs segments with a counter
// each; workgroup b appends to segment b % kFixSegs, so no single atomic
// counter serialises the K build.
constexpr int kFixSegs = 256;

enum Kind { LINEAR = 0, POLY = 1, GAUSS = 2 };

struct KappaParams {
  int kind;
  float gamma;
  float coef0;
  int degree;
  float neg_g_log2e;  // -gamma * log2(e): exp(-gamma s) = exp2(neg_g_log2e * s)
  float fix_scale;    // Gaussian: error estimate of s is fix_scale * (|x|^2 + |y|^2)
  float fix_tol;      // recompute an entry when gamma * err(s) * K exceeds this
  // The same Gaussian in terms of the scaled norms c|x|^2 (c = neg_g_log2e):
  float m2c;          // -2c: the exponent c s = m2c * (x.y) + c(|x|^2 + |y|^2)
  float fix_uthr;     // c * fix_tol / fix_scale: the fix-up test as u K < fix_uthr, u = c(|x|^2 + |y|^2)
};

// Everything a clustering iteration reads and writes on the device.
struct IterBufs {
  int64_t n, ld;
  int k, nblk, nstripes, qmax;
  int chunk_len;        // rows per SpMM chunk: kChunk, or sym_chunk_for(n) when K is packed
  int64_t col0, ncol;   // the points whose columns E^T covers: [col0, col0 + ncol)
                        // (all n from 0, except on a panel: one GPU's share)
  const float* diagK;   // n
  const double* trK;    // 1
  float* Et;            // k x ld: E transposed, E(i,j) at Et[j*ld + i]
  float* P;             // qmax x ld: per-chunk partial row sums
  double* zpart;        // k x nzpart partial self-term sums (one per reduce stripe)
  int nzpart;
  int* hist;            // k x nblk per-block cluster counts (cluster-major)
  int* base;            // k x nblk sorted position of each block's first member
  int* off;             // k + 1 cluster offsets in the sorted order
  int* qfirst;          // k + 1 first chunk of each cluster
  int* chunk_j;         // qmax
  int* chunk_p0;        // qmax
  int* chunk_p1;        // qmax
  int* nchunks;         // 1
  int* perm;            // n: sorted position -> point
  int* pos;             // n: point -> sorted position
  int* status;          // 1: bit 0 = id out of range
  // packed K only
  int nt, nseg, bseg;   // column tiles (ld / kTile); column segments of bseg tiles
  float* Ecp;           // nseg x qmax x k x chunk_len: column-side partials per segment and
                        // chunk, label-major (member t of chunk q, label j at j * chunk_len + t)
  float* Ecol;          // k x n: column-side sums, by point index
  int* chunk_c0;        // qmax: first stored column of each chunk (its first row's tile
                        // start), written by the scatter; null when K is not packed
  int* crow;            // qmax x chunk_len: point index of member t of chunk q at
                        // q * chunk_len + t (scatter); -1 past a chunk's end and at the
                        // start of an unused chunk
  unsigned* mskg;       // nt x nlb x 4 x 16 one-hot bits of each column tile (scatter):
                        // bit 4g+e of [J][nb][kk][li] says column 128J + 16g + 4kk + e
                        // has label 16nb + li
  int nlb;              // label blocks of 16, ceil(k / 16)
  const float* zero;    // kTile zero floats, read in place of rows not stored in a tile
  // stored K in binary16: entry (i, j) holds K(i,j) / kw[i] (kw null: 1);
  // packed fp32 K of the linear and polynomial kernels: kw[i] bounds
  // |K(i, .)| (null for the Gaussian)
  int kf16;
  const float* kw;
};

// binary16 storage of K
typedef _Float16 half_t;

// ---------------------------------------------------------------- launchers
hipError_t launch_stage(const float* X, int64_t n, int d, int d_pad, int64_t n_pad, float* Xp,
                        float* nrm, unsigned* maxnrm_bits, hipStream_t s);
// Row scales of binary16 storage: kw[i] bounds |K(i, j)| for every j
// (from the row norms and the largest one; linear and polynomial kernels).
hipError_t launch_row_scales(const float* nrm, const unsigned* maxnrm_bits, int64_t n, const KappaParams& kp,
                             float* kw, hipStream_t s);
// packed: store only tiles I <= J, at packed_row(i) + j (no mirror).
// f16: K is binary16, entry (i, j) stored as K(i,j) / kw[i] (kw null: 1).
// bmax[P] = the largest squared norm among points 128P .. 128P+127 of nrm
// (n_pad entries, zero past n), one per 128-point block
hipError_t launch_blockmax(const float* nrm, int64_t nblocks, float* bmax, hipStream_t s);
// bmax: the block maxima of nrm (launch_blockmax), read by the small-width
// sweep for the Gaussian kernel (may be null otherwise)
hipError_t launch_gemm_kappa(const float* Xp, const float* nrm, const unsigned* maxnrm_bits,
                             int64_t n, int d_pad, int64_t ld, bool packed, bool f16, const float* kw,
                             const KappaParams& kp, void* K, float* diagK, int2* fix_list,
                             unsigned long long* fix_count, long long seg_cap, const float* bmax, hipStream_t s);
// Recomputes the listed Gaussian entries (counts read on the device); if a
// segment received more entries than it holds, re-tests the whole triangle.
// fix_list holds kFixSegs segments of seg_cap entries; fix_count kFixSegs counters.
hipError_t launch_gauss_fixup(const float* Xp, const float* nrm, int64_t n, int d_pad, int64_t ld,
                              bool packed, bool f16, const KappaParams& kp, const int2* fix_list,
                              const unsigned long long* fix_count, long long seg_cap, void* K,
                              hipStream_t s, int64_t r0 = 0, int64_t r1 = 0, int64_t c0 = 0, int64_t c1 = 0);
// One GPU's share of a split of K: the block K[r0 : r1, c0 : c0 + ld) (r0, c0
// multiples of kTile, r1, c1 <= n, columns from c1 on stored as 0), fp32, row
// i - r0 at stride ld; diagK of the points whose diagonal the block holds;
// Gaussian entries to fix listed as (i, j), global indices
// (launch_gauss_fixup with the same r0, r1, c0, c1).  The 1D split's column
// panel is the block r0 = 0, r1 = n.
hipError_t launch_gemm_kappa_panel(const float* Xp, const float* nrm, const unsigned* maxnrm_bits,
                                   int64_t n, int d_pad, int64_t r0, int64_t r1, int64_t c0, int64_t c1,
                                   int64_t ld, const KappaParams& kp, float* K, float* diagK, int2* fix_list,
                                   unsigned long long* fix_count, long long seg_cap, hipStream_t s);
// D and lowest-index argmin for the panel's points (columns [b.col0, b.col0 + b.ncol))
// from E^T (k x ld, column = point - col0), the global z and the cluster sizes;
// counts_out gets the panel's share of the new sizes (added; zeroed by the caller).
hipError_t launch_panel_assign(const IterBufs& b, const float* z, const int* counts, int* cl_out,
                               int* counts_out, float* E_out, hipStream_t s);
// Points u < m: D(u,j) = diag[u] - 2 E(u,j)/counts[j] + z[j] over nonempty j,
// lowest-index argmin into cl_out, new sizes added to counts_out; E(u, j) at
// E[u * s_pt + j * s_cl]; E_out (nullable) gets E point-major.
hipError_t launch_cols_assign(const float* E, int64_t s_pt, int64_t s_cl, const float* diag, int64_t m, int k,
                              const float* z, const int* counts, int* cl_out, int* counts_out, float* E_out,
                              hipStream_t s);
// A piece of m points (E point-major, ids cl): per-cluster fp64 parts of
// sum_{u in L_j} E(u, j) at zpart[j * nz + g], g < ceil(m / 1024) <= nz;
// sizes added to counts; a bad id sets bit 0 of status.
hipError_t launch_cols_zpart(const float* E, const int* cl, int64_t m, int k, double* zpart, int nz, int* counts,
                             int* status, hipStream_t s);
// A block's partial E (ncol x k, point-major) from the SpMM's chunk partials.
hipError_t launch_block_out(const IterBufs& b, float* E_out, hipStream_t s);
hipError_t launch_trace(const float* diagK, int64_t n, double* trK, hipStream_t s);
// K-means++ seeding (seed.hip): one distance pass per center, one draw per
// center after the first; buffers of n (kd, D, best, bestc) and
// seed_blocks(n) (bsum) entries.
int seed_blocks(int64_t n);
hipError_t launch_kpp_dist(const float* Xp, int64_t n, int d_pad, const KappaParams& kp, int* centers, int t,
                           int c_first, float* kd, float* D, float* best, int* bestc, double* bsum, int* V,
                           hipStream_t s);
hipError_t launch_kpp_select(const float* D, const double* bsum, int64_t n, double ut, int* centers, int t,
                             hipStream_t s);
hipError_t launch_fill_diag(float* diagK, int64_t n, float v, hipStream_t s);

hipError_t launch_zero_ints(int* p, int64_t count, hipStream_t s);
// mode 0: validate cl_in, count, per-block histogram (no distances).
// mode 1: distances from Et/zpart/counts_in, argmin -> cl_out, new counts.
// counts_out must be zero on entry (scatter clears the next update's).
// pos (may be null): E^T is in sorted row order; point i reads column pos[i].
hipError_t launch_assign(int mode, const IterBufs& b, const int* counts_in, const int* cl_in,
                         const int* pos, int* cl_out, int* counts_out, int* changed, double* obj,
                         float* z_out, float* D_out, hipStream_t s);
hipError_t launch_scatter(const IterBufs& b, const int* cl, const int* counts, int* zero_counts,
                          int* zero_changed, hipStream_t s);
hipError_t launch_spmm_onehot(const void* K, const IterBufs& b, hipStream_t s);
// rows r0 .. r1-1 of a full binary16 K as fp32 (out: (r1-r0) x n)
hipError_t launch_rows_f16(const half_t* K, const float* kw, int64_t n, int64_t ld, int64_t r0, int64_t r1,
                           float* out, hipStream_t s);
hipError_t launch_spmm_reduce(const IterBufs& b, const int* cl, hipStream_t s);

// packed K (upper block triangle)
// needs the scatter's crow and mskg for the current ids
hipError_t launch_spmm_sym(const void* Kp, const IterBufs& b, hipStream_t s);
hipError_t launch_ecol_sum(const IterBufs& b, hipStream_t s);
// E^T from the chunk partials (each starting at its chunk's first stored
// column) plus the column-side sums Ecol (by point index); zpart per
// kSymRedStripe columns.
hipError_t launch_spmm_reduce_sym(const IterBufs& b, const int* cl, hipStream_t s);
hipError_t launch_packed_rows(const void* Kp, bool f16, const float* kw, int64_t n, int64_t ld, int64_t r0,
                              int64_t r1, float* out, hipStream_t s);
hipError_t launch_et_to_e(const IterBufs& b, const int* counts, const int* pos, float* E,
                          hipStream_t s);

// on-the-fly mode
struct OtfTables {
  int* cA;         // nt: first cluster of each sorted row block
  int* nruns;      // nt: clusters spanned by each block
  int64_t* cbase;  // nt: offset of each block's column-side partials (rows of 128 floats)
  float* bmax;     // nt: largest squared norm of each sorted row block
};
int onthefly_segments(int64_t n);
int64_t onthefly_cpart_floats(int64_t n, int k);
// partials per row-side and column-side entry of the sweep at this width
// (2: one per wavefront half, for the register-operand kernel of small d)
int onthefly_halves(int d_pad);
hipError_t launch_gather_sorted(const float* Xp, const float* nrm, const IterBufs& b, const int* cl,
                                int64_t n_pad, int d_pad, float* Xs, float* nrm_s, int* cs,
                                hipStream_t s);
hipError_t launch_diag_from_norms(const float* nrm, int64_t n, const KappaParams& kp, float* diagK,
                                  hipStream_t s);
hipError_t launch_onthefly(const float* Xs, const float* nrm_s, const int* cs,
                           const unsigned* maxnrm_bits, const IterBufs& b, int d_pad,
                           const KappaParams& kp, const OtfTables& tb, float* Epart, float* Cpart,
                           hipStream_t s);
hipError_t launch_onthefly_reduce(const IterBufs& b, const float* Epart, const float* Cpart,
                                  const int* cs, const OtfTables& tb, int d_pad, hipStream_t s);
hipError_t launch_kernel_rows(const float* Xp, const float* nrm, const unsigned* maxnrm_bits,
                              int64_t n, int d_pad, const KappaParams& kp, int64_t r0, int64_t r1,
                              float* out, hipStream_t s);


// Achievable-peak microbenchmarks (measurement aids, not on the clustering
// path): kPeakGrid workgroups of 256 threads stream the buffer (2040, not
// 2048, so that the workgroups' ranges do not start a power of two apart
// and their write fronts spread over the memory channels); the MFMA loop
// runs kPeakMfmaGrid workgroups of four wavefronts (four per SIMD on 256
// CUs).
constexpr int kPeakGrid = 2040;
constexpr int kPeakMfmaGrid = 1024;
hipError_t launch_peak_read(const void* buf, int64_t bytes, float* sums, hipStream_t s);
hipError_t launch_peak_write(void* buf, int64_t bytes, float value, hipStream_t s);
hipError_t launch_peak_mfma(int iters, float* out, hipStream_t s);
// nchunks x (ld / seg) workgroups of 512 threads; seg a multiple of 128
hipError_t launch_peak_rows(const float* buf, int64_t nrows, int64_t ld, const int* rows, int nchunks, int seg,
                            float* sums, hipStream_t s);

}  // namespace kkm
