/*
 * kkm.h — C ABI of the MI355X (gfx950) exact Kernel K-means engine.
 *
 * The engine computes the linear-algebraic formulation of Kernel K-means of
 * "Communication-Avoiding Linear Algebraic Kernel K-Means on GPUs"
 * (arXiv 2601.17136), Section II-B, on one GPU:
 *
 *   B = X X^T                                   (Eq. 1)
 *   K = kappa(B) elementwise                    (Eq. 2; plus linear and Gaussian)
 *   E = K V^T,  V one-hot in cluster ids        (Eq. 4, unnormalised here)
 *   z_j = (1/|L_j|^2) sum_{i in L_j} E(i,j)      (Eqs. 5-7: the paper's c_j)
 *   D(i,j) = K(i,i) - 2 E(i,j)/|L_j| + z_j       (Eq. 8 plus diag K)
 *   cl'(i) = argmin_j D(i,j)                     (end of Section II-B)
 *
 * repeated as the clustering loop of Alg. 1 with one process (every
 * collective is the identity).  V is carried as int32 cluster ids, which is
 * all the paper communicates of V (Section V).
 *
 * Conventions for every entry point:
 *  - Return value: KKM_OK (0) or a negative kkm_status.  After a failure,
 *    kkm_last_error(ctx) holds a message.  Argument checks run on the host
 *    before any HIP call; a call that fails them has enqueued nothing.
 *  - Device pointers are plain HIP device addresses (e.g. a torch tensor's
 *    data_ptr()); they stay owned by the caller.  Host pointers are marked.
 *  - Points X are n x d, fp32, row-major, contiguous (row i at X + i*d).
 *  - Cluster ids are int32 in [0, k).  An id outside that range is detected
 *    on the device and reported as KKM_ERR_DEVICE_DATA when the call
 *    synchronises; kernels clamp ids so that no access goes out of bounds.
 *    After that error the contents of every output are unspecified.
 *  - All work runs on the stream given to kkm_create.  kkm_build_kernel is
 *    asynchronous; kkm_iterate, kkm_objective, kkm_step, kkm_copy_* return
 *    after their work has completed.
 *  - A context is not thread-safe; calls on one context must not overlap.
 */
#ifndef KKM_H
#define KKM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KKM_ABI_VERSION 8
#define KKM_MAX_K 1024 /* largest supported cluster count */

typedef enum kkm_status {
  KKM_OK = 0,
  KKM_ERR_ARG = -1,         /* invalid argument; nothing enqueued */
  KKM_ERR_OOM = -2,         /* needs more device memory than the budget allows */
  KKM_ERR_HIP = -3,         /* a HIP runtime call failed (message has the HIP error) */
  KKM_ERR_STATE = -4,       /* call out of order, e.g. kkm_iterate before a build */
  KKM_ERR_DEVICE_DATA = -5  /* device input invalid: a cluster id outside [0, k) */
} kkm_status;

/* Kernel functions kappa.  LINEAR is the paper's "B = K" (Section IV);
 * POLY is Eq. 2, (gamma x.y + coef0)^degree; GAUSS is exp(-gamma |x-y|^2),
 * which the paper does not use but which the same formulation admits. */
typedef enum kkm_kind { KKM_LINEAR = 0, KKM_POLY = 1, KKM_GAUSS = 2 } kkm_kind;

/* Where K lives.  RESIDENT stores K (n*n fp32) in device memory once and
 * streams it every iteration.  PACKED stores only the upper block triangle
 * of the symmetric K (row block I of 128 rows keeps columns 128*I ..
 * ld-1, about half the bytes) and streams that: each stored entry K(i,j)
 * serves both E(j, cl(i)) and E(i, cl(j)).  PACKED handles at most
 * KKM_PACKED_MAX_K clusters and is the fastest mode up to there.  ONTHEFLY
 * never stores K: every iteration recomputes its tiles and folds them
 * straight into E, which is the paper's single-GPU sliding-window baseline
 * (Section VI-D) done tile by tile.  AUTO picks by the memory budget and
 * the cluster count the caller announces in kkm_params.k_hint:
 *   k_hint in 1..KKM_PACKED_FAST_K: PACKED if it fits, else RESIDENT if it
 *     fits, else ONTHEFLY.  PACKED's per-label column side runs on the
 *     binary16 matrix cores (an fp32 K's entries each as two binary16 parts,
 *     the rows of the linear and polynomial kernels scaled by powers of two
 *     first), which keeps it below the HBM time up to 64 labels: measured
 *     fastest there at n = 20000 .. 200000 for every kernel and storage;
 *   otherwise: RESIDENT if it fits, else (k_hint 0) PACKED if it fits, else
 *     ONTHEFLY.
 * A kkm_iterate with more than KKM_PACKED_MAX_K clusters on a K that AUTO
 * stored PACKED (k_hint 0) fails with KKM_ERR_ARG. */
typedef enum kkm_mode {
  KKM_MODE_AUTO = 0,
  KKM_MODE_RESIDENT = 1,
  KKM_MODE_ONTHEFLY = 2,
  KKM_MODE_PACKED = 3
} kkm_mode;
#define KKM_PACKED_MAX_K 64 /* largest cluster count kkm_iterate accepts on PACKED storage */
#define KKM_PACKED_FAST_K 64 /* AUTO stores K PACKED for a k_hint up to this */
#define KKM_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20) /* static scratch of kkm_iterate_noalloc, per GPU */

/* Number format of a stored K (RESIDENT or PACKED; ONTHEFLY stores nothing
 * and ignores it).  F32 keeps the fp32 entries.  F16 keeps them in IEEE
 * binary16, half the bytes to stream per iteration (mixed precision is the
 * paper's future work, Section VII): entry K(i,j) is stored as
 * fp16(K(i,j) / w_i), where w_i bounds row i (Cauchy-Schwarz:
 * |x_i . x_j| <= |x_i| max_m |x_m|; linear w_i = that bound, polynomial
 * w_i = (|gamma| * bound + |coef0|)^degree, Gaussian w_i = 1 since
 * 0 < K <= 1), so every stored value lies in [-1, 1] and keeps binary16's
 * 11 significant bits; reads multiply by w_i again and every sum runs in
 * fp32.  Each entry then carries a relative error of at most 2^-11, and
 * E(i,j) an error of at most 2^-11 sum_{m in L_j} |K(i,m)| plus the fp32
 * accumulation error; diag K, tr K, z's fp64 parts and the distances'
 * arithmetic stay fp32/fp64. */
typedef enum kkm_storage { KKM_STORE_F32 = 0, KKM_STORE_F16 = 1 } kkm_storage;

typedef struct kkm_params {
  float gamma;    /* POLY: scale of x.y; GAUSS: > 0.  Ignored for LINEAR. */
  float coef0;    /* POLY: additive constant c.  Ignored otherwise. */
  int32_t degree; /* POLY: integer exponent, 1..16.  Ignored otherwise. */
  int32_t mode;   /* kkm_mode */
  int32_t storage;/* kkm_storage of a stored K (ignored ONTHEFLY) */
  int32_t k_hint; /* clusters the loop will run with, 1..KKM_MAX_K, or 0 if not
                     known; only AUTO reads it (see kkm_mode) */
} kkm_params;

typedef struct kkm_ctx kkm_ctx; /* opaque; owns K, the staged points and all scratch */

/* Per-kernel timing, collected with HIP events on the context's stream when
 * enabled by kkm_set_timing.  Index with the KKM_PHASE_* constants. */
enum {
  KKM_PHASE_STAGE = 0,   /* copy/pad X, row norms */
  KKM_PHASE_GEMM = 1,    /* K = kappa(X X^T) tiles (resident build) */
  KKM_PHASE_FIXUP = 2,   /* Gaussian entries recomputed from differences */
  KKM_PHASE_LABELS = 3,  /* validate ids, cluster sizes, per-block counts */
  KKM_PHASE_SCATTER = 4, /* stable counting sort of points by cluster */
  KKM_PHASE_SPMM = 5,    /* E = K V^T over stored K */
  KKM_PHASE_ASSIGN = 6,  /* z, distances, argmin, new sizes */
  KKM_PHASE_ONTHEFLY = 7,/* recomputed K tiles folded into E */
  KKM_PHASE_REDUCE = 8,  /* per-cluster sums of the SpMM's chunk partials, self-term parts */
  KKM_PHASE_OTHER = 9,   /* gathers, copies, trace */
  KKM_PHASE_SEED = 10,   /* K-means++ seeding: distance passes and draws */
  KKM_NPHASE = 11
};
typedef struct kkm_timing {
  double ms[KKM_NPHASE];       /* summed kernel time per phase, milliseconds */
  int64_t launches[KKM_NPHASE];/* kernel launches per phase */
} kkm_timing;

/* Facts about the built problem. */
typedef struct kkm_info {
  int64_t n;
  int32_t d, d_pad;       /* feature count and its zero-padded width */
  int32_t kind, mode;     /* kkm_kind, resolved kkm_mode (never AUTO) */
  int32_t storage;        /* kkm_storage of K (F32 when ONTHEFLY) */
  int64_t ld;             /* RESIDENT: row stride of K in floats; PACKED: the
                             padded row length (row block I holds ld - 128*I
                             columns); ONTHEFLY: row stride of E^T */
  size_t bytes_K;         /* device bytes held by K (0 on the fly) */
  size_t bytes_total;     /* device bytes held by the context */
  int64_t fixups;         /* Gaussian entries flagged for recomputation at build */
  int64_t fixup_capacity; /* entries the fix-up list holds; beyond it the whole
                             triangle is re-tested instead */
  int64_t r0, r1, c0, c1; /* the stored rows [r0, r1) and columns [c0, c1) of K:
                             a panel or block (kkm_build_panel, kkm_build_block),
                             else 0, n, 0, n */
} kkm_info;

/* Create a context on the current HIP device.
 * out:        receives the context (host pointer).
 * hip_stream: hipStream_t to run on; NULL = the default (null) stream.
 * mem_budget: device bytes the context may hold; 0 = 95% of the free memory
 *             reported by hipMemGetInfo at creation.
 * Errors: KKM_ERR_ARG (out NULL), KKM_ERR_HIP. */
int kkm_create(kkm_ctx **out, void *hip_stream, size_t mem_budget);

/* Free every device buffer the context holds, then the context.  NULL is a no-op. */
int kkm_destroy(kkm_ctx *ctx);

/* Message describing the last failure on ctx ("" if none).  With ctx NULL,
 * the last failure of a call that had no context (kkm_create, kkm_plan). */
const char *kkm_last_error(const kkm_ctx *ctx);

/* Warning of the last build on ctx ("" if none); with ctx NULL, of the last
 * kkm_check_build_args on the calling thread.  A build that warns still
 * succeeds.  The one warning: a polynomial kernel with coef0 < 0 or
 * gamma < 0 is not positive semidefinite (Eq. 2 with integer degree is PSD
 * only for gamma, coef0 >= 0), so K may have negative eigenvalues and the
 * objective need not fall from update to update. */
const char *kkm_last_warning(const kkm_ctx *ctx);

/* Pure host planning, no HIP call.  Picks the mode for a problem and the
 * device bytes it needs (K, staged points, per-iteration scratch for k
 * clusters).  A context created with that many bytes builds and iterates:
 * the Gaussian build's fix-up list takes up to a quarter of the room the
 * budget leaves, and the first iteration that needs that room frees it
 * (after one synchronisation to read its counts), so it is not counted
 * here.  kind: kkm_kind of the kernel to be built (the linear and
 * polynomial kernels keep a bound per row where K is packed or binary16).
 * requested_mode: kkm_mode; AUTO resolves by the budget and k as a build
 * with k_hint = k does (see kkm_mode).
 * storage: kkm_storage of K (sizes K and the row bounds).
 * Errors: KKM_ERR_ARG (bad sizes, kind or storage, or PACKED with
 * k > KKM_PACKED_MAX_K), KKM_ERR_OOM (even the on-the-fly mode does not fit,
 * or the requested storing mode does not). */
int kkm_plan(int64_t n, int32_t d, int32_t k, int32_t kind, size_t mem_budget, int32_t requested_mode,
             int32_t storage, int32_t *mode_out, size_t *bytes_out);

/* Host-only argument checks that the entry points apply first; exported so
 * they can be exercised without a GPU.  Return KKM_OK or KKM_ERR_ARG;
 * kkm_check_build_args also sets the warning kkm_last_warning(NULL) reads. */
int kkm_check_build_args(int64_t n, int32_t d, int32_t kind, const kkm_params *params);
int kkm_check_iterate_args(int64_t n, int32_t k, int32_t max_iter);

/* Build the kernel matrix K = kappa(X X^T) (Eqs. 1-2) for the clustering loop.
 * X:      device, n x d fp32 row-major.  The engine copies it (zero-padded to
 *         d_pad columns); the caller may free X once this call has returned.
 * n:      points, 1 .. 2^31-1.   d: features, 1 .. 65536.
 * kind:   kkm_kind.   params: host pointer (gamma, coef0, degree, mode, storage,
 *         k_hint).
 * RESIDENT: stores K (n rows, stride ld) in device memory; diag K is exact
 *   (Gaussian: exactly 1).  Gaussian entries whose expansion
 *   |x|^2 + |y|^2 - 2 x.y may have lost accuracy to cancellation are
 *   recomputed from the coordinate differences.
 * PACKED: as RESIDENT, but only the tiles I <= J of the 128 x 128 tiling
 *   are stored (row i keeps columns 128*floor(i/128) .. ld-1).  The linear
 *   and polynomial kernels also keep a bound per row (Cauchy-Schwarz) for
 *   the update's column side, which sums each fp32 entry's two binary16
 *   parts: an entry v of row i is represented within
 *   max(2^-22 |v|, 2^-25 p_i), p_i the power of two at or above the bound
 *   (1 for the Gaussian), and every sum stays fp32.
 * ONTHEFLY: stages X and row norms only.
 * storage F16 (RESIDENT, PACKED): K in binary16 with row scales, see
 *   kkm_storage; diag K stays fp32.
 * Replaces any earlier build on ctx; a build of the same n, d, kind and mode
 * reuses the device buffers of the previous one.  Asynchronous.
 * Errors: KKM_ERR_ARG, KKM_ERR_OOM, KKM_ERR_HIP. */
int kkm_build_kernel(kkm_ctx *ctx, const float *X, int64_t n, int32_t d, int32_t kind,
                     const kkm_params *params);

/* Run the clustering loop (Alg. 1 with one process).
 * V:          device int32[n]: the initial cluster ids on entry, the final
 *             ids on return.
 * k:          clusters, 1 .. min(n, KKM_MAX_K); at most KKM_PACKED_MAX_K
 *             when K was built PACKED.
 * max_iter:   >= 0 assignment updates at most.
 * tol:        < 0: run exactly max_iter updates (no host round trip per
 *             update).  = 0: stop after an update that changed no id.
 *             > 0: also stop once J(prev) - J(cur) <= tol * |J(prev)|.
 * iters_done: host, may be NULL: updates applied.
 * obj_hist:   host, may be NULL, max_iter entries: obj_hist[t] = J(cl_t),
 *             the objective sum_i D(i, cl_t(i)) of the ids before update t.
 * Empty clusters get D = +inf (never chosen) and stay empty; ties go to the
 * lowest cluster index.
 * Errors: KKM_ERR_ARG, KKM_ERR_STATE (no build), KKM_ERR_DEVICE_DATA, KKM_ERR_OOM, KKM_ERR_HIP. */
int kkm_iterate(kkm_ctx *ctx, int32_t *V, int32_t k, int32_t max_iter, double tol,
                int32_t *iters_done, double *obj_hist);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): kkm_iterate
 * with the same arguments, results and errors, whose per-update scratch and
 * objective history live in a static device array of
 * KKM_NOALLOC_SCRATCH_BYTES per GPU (allocated when the library's code is
 * loaded on that GPU, held until the process ends) instead of buffers the
 * context allocates.  It calls no hipMalloc or hipFree; the K and staged
 * points of the build are the context's.  Problems whose scratch does not fit
 * (for example n = 20000 with packed K and k = 10 needs about 45 MB, with the
 * full K about 4 MB) fail with KKM_ERR_ARG before anything is enqueued.  Every call
 * on a GPU shares that GPU's array and leaves its contents behind: calls
 * that overlap on one GPU (other threads, streams or contexts) race, so the
 * caller serializes them.  No launch is bracketed by timing events.
 * The context's own scratch, if an earlier kkm_iterate made one, is left as
 * it was. */
int kkm_iterate_noalloc(kkm_ctx *ctx, int32_t *V, int32_t k, int32_t max_iter, double tol,
                        int32_t *iters_done, double *obj_hist);

/* J(cl) = sum_i D(i, cl(i)) = tr K - sum_j |L_j| z_j for the ids V (device
 * int32[n]); written to *J (host).  Errors as kkm_iterate. */
int kkm_objective(kkm_ctx *ctx, const int32_t *V, int32_t k, double *J);

/* One clustering step from ids cl_in, exposing every intermediate (for
 * parity checks; not tuned).  All pointers are device memory except J.
 * E: n x k fp32 row-major, E(i,j) = sum_{m: cl(m)=j} K(i,m)  (may be NULL)
 * z: k fp32, the cluster self-terms                          (may be NULL)
 * D: n x k fp32 row-major distances, +inf for empty clusters (may be NULL)
 * cl_out: n int32 new ids; counts_out: k int32 sizes of cl_in (may be NULL each)
 * J: host double, J(cl_in)                                   (may be NULL)
 * Errors as kkm_iterate. */
int kkm_step(kkm_ctx *ctx, const int32_t *cl_in, int32_t k, float *E, float *z, float *D,
             int32_t *cl_out, int32_t *counts_out, double *J);

/* K-means++ seeding in the kernel's feature space (the initialization the
 * paper cites for its convergence properties in Section II-B and leaves to
 * future work in Section V): D^2 sampling of k centers among the points,
 * then each point's nearest center as its initial id.
 *   u[0]      picks the first center, floor(u[0] * n);
 *   D(i)      = min over chosen centers c of K(i,i) - 2 K(i,c) + K(c,c);
 *   center t  = the first index i with sum_{m <= i} D(m) > u[t] * sum_m D(m),
 *               i.e. i with probability D(i) / sum D; if the sum is 0 (every
 *               point coincides with a chosen center), the lowest index not
 *               yet chosen.
 * The entries of K are computed from the staged points of the last build,
 * in every storage mode (the Gaussian from the coordinate differences).
 * u:           host, k doubles in [0, 1), the caller's uniforms (the draws
 *              are reproducible from them).
 * centers_out: host, may be NULL, k int32: the chosen point indices in order.
 * V:           device int32[n], written with the position (0 .. k-1) in the
 *              center list of each point's nearest center, lowest position
 *              among equal distances: ready for kkm_iterate.
 * Sums run in a fixed order in fp64 over fp32 distances, so results are
 * reproducible.  The context allocates O(n) scratch on first use.
 * Synchronises before returning.
 * Errors: KKM_ERR_ARG (k outside 1..min(n, KKM_MAX_K), u NULL or outside
 * [0, 1), V NULL), KKM_ERR_STATE (no build), KKM_ERR_OOM, KKM_ERR_HIP. */
int kkm_init_kmeanspp(kkm_ctx *ctx, int32_t k, const double *u, int32_t *centers_out, int32_t *V);

/* One GPU's share of the 1D split (the paper's 1D algorithm, Section IV-A,
 * Algorithm 1: each process holds the column block of K for its points and
 * the ids of all points).  GPU g of G owns the points [c0, c1) and holds the
 * column panel K[:, c0:c1], all n rows.  Per update:
 *   kkm_panel_spmm    E(i, j) = sum_{m: cl(m)=j} K(i, m) for its points i
 *                     (kept in the context) and its part of the self-terms,
 *                     zpart_j = sum_{i in [c0,c1), cl(i)=j} E(i, j);
 *   (exchange)        the caller sums zpart over the G GPUs (an all-reduce of
 *                     k doubles) and forms z_j = sum_g zpart_j / |L_j|^2;
 *   kkm_panel_assign  D(i, j) = K(i,i) - 2 E(i,j)/|L_j| + z_j and the new ids
 *                     of its points (lowest index on ties, +inf for empty j);
 *   (exchange)        the caller gathers the new ids of all points (an
 *                     all-gather of 4n bytes) for the next update.
 * The exchanges are not part of the library.
 *
 * kkm_build_panel: as kkm_build_kernel (params->mode is ignored; storage must
 * be KKM_STORE_F32) for the panel of points [c0, c1): 0 <= c0 < c1 <= n, c0
 * a multiple of 128, c1 - c0 <= 8,388,480 (the K build addresses a tile's
 * stores with 32-bit offsets).  The panel takes n x round_up(c1 - c0, 128) floats; its
 * tiles are computed whole (no symmetry saving), the Gaussian diagonal is 1
 * and flagged Gaussian entries are recomputed from the differences, as in
 * the full build.  Only the panel's points get diag K.  After it,
 * kkm_copy_kernel_rows copies rows of the panel ((r1-r0) x (c1-c0)), and
 * kkm_iterate, kkm_step and kkm_objective return KKM_ERR_STATE.
 * Errors: KKM_ERR_ARG (as kkm_build_kernel, a bad range, fp16 storage),
 * KKM_ERR_OOM, KKM_ERR_HIP. */
int kkm_build_panel(kkm_ctx *ctx, const float *X, int64_t n, int32_t d, int32_t kind,
                    const kkm_params *params, int64_t c0, int64_t c1);

/* cl: device int32[n], the ids of all points.  zpart: host, k doubles (the
 * sum over the SpMM's column stripes in order).  counts: host, may be NULL, k
 * int32: |L_j| over all n points.  Synchronises before returning.
 * Errors: KKM_ERR_ARG, KKM_ERR_STATE (no panel built), KKM_ERR_DEVICE_DATA
 * (an id outside [0, k)), KKM_ERR_OOM, KKM_ERR_HIP. */
int kkm_panel_spmm(kkm_ctx *ctx, const int32_t *cl, int32_t k, double *zpart, int32_t *counts);

/* z: host, k doubles, the global self-terms (converted to fp32 as the full
 * step uses them).  cl_out: device int32[c1 - c0], the new ids of the points
 * c0 .. c1-1.  E_out: device, may be NULL, (c1 - c0) x k fp32 row-major, the
 * panel's rows of E.  counts_out: host, may be NULL, k int32: how many of the
 * panel's points took each id.  Uses the sizes and E of the last
 * kkm_panel_spmm, which must have had the same k.  Synchronises before
 * returning.  Errors: KKM_ERR_ARG, KKM_ERR_STATE, KKM_ERR_HIP. */
int kkm_panel_assign(kkm_ctx *ctx, int32_t k, const double *z, int32_t *cl_out, float *E_out,
                     int32_t *counts_out);

/* One GPU's share of the 1.5D split (the paper's 1.5D algorithm, Section
 * IV-C, Algorithm 2: K is computed by SUMMA and stays 2D-partitioned over a
 * sqrt(P) x sqrt(P) process grid; V stays 1D-partitioned).  The points are
 * cut into sqrt(P) contiguous blocks, and each block into sqrt(P) pieces
 * (the 1D partition, P pieces in all).  Process (i, j) holds the block
 * K[rows of block i, columns of block j] and owns piece l = i of column
 * block j.  Per update:
 *   (exchange)        the caller gathers the ids of row block i on each
 *                     process of grid row i (an all-gather along the row);
 *   kkm_block_spmm    the partial E(u, j') = sum over the block's rows r with
 *                     cl(r) = j' of K(r, u), for its columns u;
 *   (exchange)        the caller sums the partials of grid column j and
 *                     splits them by columns (a reduce-scatter along the
 *                     column): each process gets E of its own piece;
 *   kkm_block_zpart   its piece's part of the self-terms and its sizes;
 *   (exchange)        the caller sums both over all processes (an
 *                     all-reduce of k doubles and k ints) and forms
 *                     z_j = sum zpart_j / |L_j|^2;
 *   kkm_block_assign  D(u, j) = K(u,u) - 2 E(u,j)/|L_j| + z_j and the new ids
 *                     of its piece (lowest index on ties, +inf for empty j).
 * The ids of a piece are the process's own part of V; the exchanges are not
 * part of the library.  The 1D split's panel is the block of all rows
 * (kkm_build_panel); these calls also run on it.
 *
 * kkm_build_block: as kkm_build_panel for the block rows [r0, r1) x columns
 * [c0, c1): 0 <= r0 < r1 <= n and 0 <= c0 < c1 <= n, r0 and c0 multiples of
 * 128, c1 - c0 <= 8,388,480 (as for a panel).  The block takes
 * (r1 - r0) x round_up(c1 - c0, 128) floats.  diag K is
 * set for every point, from the staged norms (Gaussian: 1).  A rebuild with
 * blocks of the same size keeps the buffers.  After it, kkm_copy_kernel_rows
 * copies rows r0 <= r < r1 of the block ((r1-r0) x (c1-c0)); the full-K and
 * panel calls return KKM_ERR_STATE.
 * Errors: KKM_ERR_ARG (as kkm_build_kernel, a bad range, fp16 storage),
 * KKM_ERR_OOM, KKM_ERR_HIP. */
int kkm_build_block(kkm_ctx *ctx, const float *X, int64_t n, int32_t d, int32_t kind,
                    const kkm_params *params, int64_t r0, int64_t r1, int64_t c0, int64_t c1);

/* cl: device int32[r1 - r0], the ids of the block's rows r0 .. r1-1.  E_out:
 * device, (c1 - c0) x k fp32 row-major (point-major, so that the columns of a
 * piece are contiguous for the reduce-scatter): E_out[u*k + j] = sum over
 * r in [r0, r1) with cl[r - r0] = j of K(r, c0 + u), 0 for an id no row
 * holds; summed in a fixed order.  Synchronises before returning.
 * Errors: KKM_ERR_ARG, KKM_ERR_STATE (no block built), KKM_ERR_DEVICE_DATA
 * (an id outside [0, k)), KKM_ERR_OOM, KKM_ERR_HIP. */
int kkm_block_spmm(kkm_ctx *ctx, const int32_t *cl, int32_t k, float *E_out);

/* The piece [a0, a1) of the block's columns (c0 <= a0 < a1 <= c1).  E:
 * device, (a1 - a0) x k fp32 row-major, the piece's rows of E (the summed
 * partials); cl: device int32[a1 - a0], the piece's ids.  zpart: host, k
 * doubles, zpart_j = sum_{u in piece, cl(u)=j} E(u, j) (fp64, fixed order).
 * counts: host, k int32, the piece's cluster sizes.  Synchronises before
 * returning.  Errors: KKM_ERR_ARG (range, NULL), KKM_ERR_STATE,
 * KKM_ERR_DEVICE_DATA (an id outside [0, k)), KKM_ERR_OOM, KKM_ERR_HIP. */
int kkm_block_zpart(kkm_ctx *ctx, const float *E, const int32_t *cl, int64_t a0, int64_t a1, int32_t k,
                    double *zpart, int32_t *counts);

/* The piece [a0, a1) as in kkm_block_zpart, E as there.  z: host, k doubles,
 * the global self-terms (converted to fp32 as the full step uses them);
 * counts: host, k int32, the global sizes |L_j| (>= 0).  cl_out: device
 * int32[a1 - a0], the piece's new ids.  counts_out: host, may be NULL, k
 * int32: how many of the piece's points took each id.  Synchronises before
 * returning.  Errors: KKM_ERR_ARG (range, NULL, a negative size),
 * KKM_ERR_STATE, KKM_ERR_OOM, KKM_ERR_HIP. */
int kkm_block_assign(kkm_ctx *ctx, const float *E, int64_t a0, int64_t a1, int32_t k, const double *z,
                     const int32_t *counts, int32_t *cl_out, int32_t *counts_out);

/* Rows r0 .. r1-1 of K into out (device, (r1-r0) x n fp32 row-major).  In
 * ONTHEFLY mode the rows are computed by the same tile kernel the loop uses;
 * in PACKED mode the part left of the stored triangle is read by symmetry.
 * Errors: KKM_ERR_ARG (range), KKM_ERR_STATE, KKM_ERR_HIP. */
int kkm_copy_kernel_rows(kkm_ctx *ctx, int64_t r0, int64_t r1, float *out);

/* diag K into out (device, n fp32). */
int kkm_copy_diag(kkm_ctx *ctx, float *out);

/* Timing: phase_mask selects the phases whose kernel launches are bracketed
 * by HIP events on the context's stream (bit 1 << KKM_PHASE_x; KKM_TIME_ALL
 * for every phase; 0 disables timing).  Each bracket costs a few
 * microseconds of stream time, so time only the kernels of interest in a
 * measured run.  Setting a mask also clears the accumulated figures.
 * kkm_get_timing synchronises the stream and returns the sums so far. */
#define KKM_TIME_ALL ((1 << KKM_NPHASE) - 1)
int kkm_set_timing(kkm_ctx *ctx, int32_t phase_mask);
int kkm_get_timing(kkm_ctx *ctx, kkm_timing *out);

int kkm_get_info(kkm_ctx *ctx, kkm_info *out);

/* Achievable-peak microbenchmarks.  These are measurement aids and no step of
 * the method: they give what this GPU sustains, so the roofline fractions of
 * the kernels above can be stated against measured peaks as well as the
 * datasheet ones.  Each runs reps launches of one kernel on the context's
 * stream and writes the average launch time in ms to *ms_out (host); it
 * returns after the launches have completed.  Errors: KKM_ERR_ARG (NULL
 * pointers, bytes not a positive multiple of 16, a buffer not 16-byte
 * aligned, reps or iters < 1; for kkm_peak_read_rows also nrows < 1, ld not
 * a multiple of 4 or below 128, seg not a positive multiple of 128 or above
 * ld, nchunks < 1, or more than 2^32 - 1 work-items in the launch),
 * KKM_ERR_HIP.
 *  - kkm_peak_read: non-temporal 16-byte loads over buf (device, `bytes`
 *    bytes read as fp32), 2040 workgroups, each streaming a contiguous
 *    range 16 KB at a time; workgroup g writes the fp32 sum
 *    of the values it read to sums[g] (device, at least 2040 floats), so
 *    the loads cannot be elided and the caller can check them.
 *  - kkm_peak_write: non-temporal 16-byte stores of `value` over buf.
 *  - kkm_peak_read_rows: the packed SpMM's load pattern without its
 *    arithmetic, so its rate can be stated against what the pattern itself
 *    sustains.  buf (device) is an nrows x ld fp32 matrix, row-major (ld a
 *    multiple of 4, at least 128); rows (device) holds nchunks x 128 row
 *    indices, clamped into [0, nrows) when read.  Workgroup (c, s), for
 *    c < nchunks and s < ld / seg (seg a multiple of 128, at most ld), reads
 *    rows rows[128c .. 128c + 127] over columns [s*seg, (s+1)*seg): eight
 *    wavefronts of 16 rows, each step 128 columns of its rows with
 *    non-temporal 16-byte loads (two rows of 512 contiguous bytes per
 *    instruction), one step in flight per wavefront.  It writes the fp32
 *    sum of what it read to sums[c * (ld / seg) + s] (device, that many
 *    floats).  Bytes read per launch: nchunks * 128 * (ld / seg) * seg * 4.
 *  - kkm_peak_mfma: four independent chains of v_mfma_f32_32x32x2_f32 per
 *    wavefront, `iters` instructions each, 1024 workgroups of four
 *    wavefronts; one float per wavefront to out (device, at least 4096
 *    floats); *flops_out (host) = the fp32 matrix flop of one launch. */
int kkm_peak_read(kkm_ctx *ctx, const void *buf, size_t bytes, float *sums, int32_t reps, float *ms_out);
int kkm_peak_write(kkm_ctx *ctx, void *buf, size_t bytes, float value, int32_t reps, float *ms_out);
int kkm_peak_read_rows(kkm_ctx *ctx, const void *buf, int64_t nrows, int64_t ld, const int32_t *rows,
                       int32_t nchunks, int32_t seg, float *sums, int32_t reps, float *ms_out);
int kkm_peak_mfma(kkm_ctx *ctx, int32_t iters, float *out, int32_t reps, float *ms_out, double *flops_out);

int kkm_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* KKM_H */
