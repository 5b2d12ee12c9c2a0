/* Sanitizer driver for the oracle's C Householder QR: factors a few matrices
 * (including n = 1, a zero column and a rank-deficient one) and checks the
 * fp64 residuals.  Exits 0 on success. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_householder_qr(int64_t n, const double *A, double *Q, double *R, int nthreads);

static double resid(int64_t n, const double *A, const double *Q, const double *R, double *orth) {
  double num = 0, den = 0, o = 0;
  for (int64_t i = 0; i < n; ++i)
    for (int64_t j = 0; j < n; ++j) {
      double s = 0, t = 0;
      for (int64_t k = 0; k < n; ++k) {
        s += Q[i * n + k] * R[k * n + j];
        t += Q[k * n + i] * Q[k * n + j];
      }
      num += (s - A[i * n + j]) * (s - A[i * n + j]);
      den += A[i * n + j] * A[i * n + j];
      t -= (i == j);
      o += t * t;
    }
  *orth = sqrt(o / (double)n);
  return den > 0 ? sqrt(num / den) : sqrt(num);
}

int main(void) {
  const int64_t sizes[] = {1, 2, 7, 33, 130};
  int bad = 0;
  unsigned s = 12345u;
  for (int c = 0; c < 5; ++c) {
    const int64_t n = sizes[c];
    double *A = malloc(sizeof(double) * n * n), *Q = malloc(sizeof(double) * n * n),
           *R = malloc(sizeof(double) * n * n);
    for (int64_t i = 0; i < n * n; ++i) {
      s = s * 1103515245u + 12345u;
      A[i] = ((double)(s >> 8) / 16777216.0) - 0.5;
    }
    if (n > 3) {            /* a zero column and a repeated one */
      for (int64_t i = 0; i < n; ++i) { A[i * n + 1] = 0.0; A[i * n + 3] = A[i * n + 2]; }
    }
    double orth = 0;
    if (oracle_householder_qr(n, A, Q, R, 2) != 0) { printf("FAIL qr n=%lld\n", (long long)n); ++bad; }
    const double r = resid(n, A, Q, R, &orth);
    if (!(r <= 1e-12) || !(orth <= 1e-12)) { printf("FAIL n=%lld resid %g orth %g\n", (long long)n, r, orth); ++bad; }
    free(A); free(Q); free(R);
  }
  if (oracle_householder_qr(0, NULL, NULL, NULL, 1) != -1) { printf("FAIL n=0 accepted\n"); ++bad; }
  printf("%s\n", bad ? "FAILED" : "ok");
  return bad ? 1 : 0;
}
