/*
 * fp64 textbook Householder QR for the SOAP oracle.
 *
 * TEST INFRASTRUCTURE ONLY: this file belongs to the CPU oracle that checks the
 * HIP path.  Only tests/, the smoke check and the bench's CPU-baseline leg may
 * load it.  It shares no code with the HIP library.
 *
 * What it computes (the paper's eigenbasis refresh, SOAP Alg. 2, takes
 * "QR(L Q_L).Q" and "QR(R Q_R).Q"): the Q factor of A = QR with the diagonal
 * of R made non-negative, which is unique for nonsingular A.
 *
 * Algorithm (Householder triangularisation, column by column, unblocked):
 *   for k = 0 .. n-1:
 *     x = A[k:, k];  if ||x[1:]|| == 0 the column is already triangular: H_k = I
 *     sigma = ||x||;  alpha = -sgn(x0) * sigma with sgn(0) = +1
 *     v = x - alpha e_1;  A[k:, k:] -= (2 / v^T v) v (v^T A[k:, k:])
 *   R = triu(A);  Q = H_0 H_1 ... H_{n-1} applied to I from the last reflector back
 *   for each k with R[k,k] < 0: negate column k of Q and row k of R.
 * Arithmetic is plain fp64 with sums in increasing row order.  The only
 * parallelism is over independent columns of each rank-1 update (OpenMP), which
 * does not change any individual sum.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Apply H = I - s v v^T to columns [c0, n) of the column-major block whose
 * column j starts at col(j) + r0, rows r0 .. r0+len-1. */
static void apply_reflector(double *a, int64_t n, int64_t r0, int64_t c0,
                            const double *v, int64_t len, double s) {
  int64_t ncols = n - c0;
#pragma omp parallel for schedule(static) if (ncols * len > 65536)
  for (int64_t jj = 0; jj < ncols; ++jj) {
    double *col = a + (c0 + jj) * n + r0;
    double w = 0.0;
    for (int64_t i = 0; i < len; ++i) w += v[i] * col[i];
    double f = s * w;
    for (int64_t i = 0; i < len; ++i) col[i] -= f * v[i];
  }
}

/* A, Q, R: n x n row-major fp64.  A is not modified.  R may be NULL.
 * Returns 0 on success, -1 on allocation failure or bad n. */
int oracle_householder_qr(int64_t n, const double *A, double *Q, double *R,
                          int nthreads) {
  if (n < 1) return -1;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
  double *a = (double *)malloc(sizeof(double) * n * n);   /* column-major work copy */
  double *q = (double *)malloc(sizeof(double) * n * n);
  double *vs = (double *)malloc(sizeof(double) * n * n);  /* v_k stored at vs[k*n + k ..] */
  double *sc = (double *)malloc(sizeof(double) * n);       /* 2 / v^T v, or 0 for H = I */
  if (!a || !q || !vs || !sc) { free(a); free(q); free(vs); free(sc); return -1; }
  for (int64_t i = 0; i < n; ++i)
    for (int64_t j = 0; j < n; ++j) a[j * n + i] = A[i * n + j];

  for (int64_t k = 0; k < n; ++k) {
    double *x = a + k * n + k;
    int64_t len = n - k;
    double tail = 0.0;
    for (int64_t i = 1; i < len; ++i) tail += x[i] * x[i];
    if (tail == 0.0) { sc[k] = 0.0; continue; }           /* H_k = I */
    double sigma = sqrt(x[0] * x[0] + tail);
    double alpha = (x[0] >= 0.0) ? -sigma : sigma;
    double *v = vs + k * n + k;
    for (int64_t i = 0; i < len; ++i) v[i] = x[i];
    v[0] -= alpha;
    double vtv = 0.0;
    for (int64_t i = 0; i < len; ++i) vtv += v[i] * v[i];
    sc[k] = 2.0 / vtv;
    apply_reflector(a, n, k, k, v, len, sc[k]);
  }

  for (int64_t j = 0; j < n; ++j)
    for (int64_t i = 0; i < n; ++i) q[j * n + i] = (i == j) ? 1.0 : 0.0;
  for (int64_t k = n - 1; k >= 0; --k) {
    if (sc[k] == 0.0) continue;
    apply_reflector(q, n, k, k, vs + k * n + k, n - k, sc[k]);
  }

  for (int64_t k = 0; k < n; ++k) {
    double d = a[k * n + k];
    double sgn = (d < 0.0) ? -1.0 : 1.0;
    for (int64_t i = 0; i < n; ++i) Q[i * n + k] = sgn * q[k * n + i];
    if (R) {
      for (int64_t j = 0; j < n; ++j)
        R[k * n + j] = (j >= k) ? sgn * a[j * n + k] : 0.0;
    }
  }
  free(a); free(q); free(vs); free(sc);
  return 0;
}
