/*
 * Oracle kernel-function evaluator (TEST INFRASTRUCTURE ONLY).
 *
 * Evaluates entries of the kernel matrix K(i,j) = kappa(x_i, x_j) straight
 * from the definition of each kernel function, in double precision, from the
 * single-precision points the engine also receives:
 *
 *   linear      kappa(x,y) = x.y                  (Section IV: "B = K")
 *   polynomial  kappa(x,y) = (gamma x.y + c)^p    (Section II-B, Eq. 2; the
 *                                                 paper writes the exponent d)
 *   Gaussian    kappa(x,y) = exp(-gamma |x-y|^2)  (not in the paper; the squared
 *                                                 distance is summed from the
 *                                                 coordinate differences, never
 *                                                 from norms and dot products)
 *
 * Nothing here is shared with the GPU engine; only the Python oracle module in
 * this directory loads it, and only tests, the smoke check and the benchmark's
 * CPU-baseline leg call that module.
 */
#include <math.h>
#include <stdint.h>

enum { REF_LINEAR = 0, REF_POLY = 1, REF_GAUSS = 2 };

static double ref_kappa(const float *x, const float *y, int32_t d, int32_t kind,
                        double gamma, double coef0, int32_t degree) {
  if (kind == REF_GAUSS) {
    double s = 0.0;
#pragma omp simd reduction(+ : s)
    for (int32_t t = 0; t < d; t++) {
      double diff = (double)x[t] - (double)y[t];
      s += diff * diff;
    }
    return exp(-gamma * s);
  }
  double dot = 0.0;
#pragma omp simd reduction(+ : dot)
  for (int32_t t = 0; t < d; t++) dot += (double)x[t] * (double)y[t];
  if (kind == REF_LINEAR) return dot;
  double base = gamma * dot + coef0, v = 1.0;
  for (int32_t e = 0; e < degree; e++) v *= base; /* integer exponent */
  return v;
}

/* out[a*nc + b] = kappa(X[rows[a]], X[cols[b]]); X is n x d row-major fp32. */
void kkm_ref_kernel_block(const float *X, int64_t n, int32_t d, int32_t kind,
                          double gamma, double coef0, int32_t degree,
                          const int64_t *rows, int64_t nr,
                          const int64_t *cols, int64_t nc, double *out) {
  (void)n;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t a = 0; a < nr; a++) {
    const float *x = X + rows[a] * (int64_t)d;
    double *o = out + a * nc;
    for (int64_t b = 0; b < nc; b++)
      o[b] = ref_kappa(x, X + cols[b] * (int64_t)d, d, kind, gamma, coef0, degree);
  }
}

/* out[p] = kappa(X[rows[p]], X[cols[p]]) for p < np_: single entries, e.g. the
 * diagonal K(i,i) or sampled entries of a matrix too large to form. */
void kkm_ref_kernel_pairs(const float *X, int64_t n, int32_t d, int32_t kind,
                          double gamma, double coef0, int32_t degree,
                          const int64_t *rows, const int64_t *cols, int64_t np_,
                          double *out) {
  (void)n;
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < np_; p++)
    out[p] = ref_kappa(X + rows[p] * (int64_t)d, X + cols[p] * (int64_t)d, d,
                       kind, gamma, coef0, degree);
}

/*
 * own[a] = sum over members m of cluster cl[rows[a]] of kappa(x_rows[a], x_m):
 * the per-point mask value z(i) = E(i, cl(i)) of Eq. 5 with an unnormalised
 * one-hot V, needed for the cluster self-terms of Eq. 6 without forming all of
 * K.  members/offsets list the points of each cluster (CSR by cluster).
 */
void kkm_ref_own_cluster_sums(const float *X, int64_t n, int32_t d, int32_t kind,
                              double gamma, double coef0, int32_t degree,
                              const int32_t *cl, const int64_t *members,
                              const int64_t *offsets, const int64_t *rows,
                              int64_t nr, double *own) {
  (void)n;
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t a = 0; a < nr; a++) {
    int64_t i = rows[a];
    int32_t j = cl[i];
    const float *x = X + i * (int64_t)d;
    double s = 0.0;
    for (int64_t q = offsets[j]; q < offsets[j + 1]; q++)
      s += ref_kappa(x, X + members[q] * (int64_t)d, d, kind, gamma, coef0, degree);
    own[a] = s;
  }
}

int kkm_ref_abi_version(void) { return 1; }
